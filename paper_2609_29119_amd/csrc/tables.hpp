// Device-visible table records shared by the host plan builder and the HIP
// kernels. Plain structs only: the host fills them in fp64 and stores fp32.
#pragma once

#include <cstdint>

namespace nsg {

// Largest prime radix of a Stockham stage. Primes above 16 run on the matrix
// cores, which form the stage's outputs as products with the cosine and sine
// matrices of the prime. Band lengths with a larger prime factor, or whose
// stage does not fit a workgroup's matrix tiles, are transformed with
// Bluestein's chirp-z algorithm over a length P >= 2M - 1 with prime factors
// up to 13, which is also used where the cost model finds it cheaper.
constexpr int kMfmaMaxRadix = 257;
constexpr int kMaxStages = 24;
// 16 x 16 result tiles one wave keeps in registers across the barrier of a
// matrix-core stage.
constexpr int kMfmaTilesPerWave = 4;

// Result tiles of a matrix-core stage of prime radix R over totb butterfly
// columns: blocks of 8 complex columns times blocks of 16 outputs q = 0..(R-1)/2.
inline constexpr int mfma_tiles(int totb, int R) { return ((totb + 7) >> 3) * (((R - 1) / 2 + 16) >> 4); }

// One transform length n: Stockham stages of the given radices, applied in
// order. Twiddle pool layout per length: the full table omega_n^t (t < n) at
// `full`, the two-level table (hi: nhi values, lo: 2^lg values) right after
// it, and the stage twiddles at `stw`: for stage s >= 1 with radix R over
// Ns = product of the earlier radices, omega_{Ns R}^{r k} at
// stw + stoff[s] + k (R - 1) + r - 1 for k < Ns, 1 <= r < R (ntw values in all).
struct FftDesc {
    int32_t n;
    int32_t nstages;
    int32_t full;
    int32_t lg;
    int32_t nhi;
    int32_t stw;
    int32_t ntw;
    int16_t radix[kMaxStages];
    int32_t stoff[kMaxStages];
    // per stage: 1 / Ns (the product of the earlier radices) and, for a prime
    // radix R > 16, 1 / ((R - 1) / 2), rounded once to fp32; the stages'
    // quotient-and-remainder steps start from these (see Div)
    float rcp_ns[kMaxStages];
    float rcp_h[kMaxStages];
};

// One band of the layout as the band kernels see it.
struct BandDev {
    int32_t k_lo;      // first support bin
    int32_t M;         // band length, at least the support width
    int32_t W;         // support width: entries i < W hold bins k_lo + i
    int32_t rot;       // slot of bin k_lo: (k_lo - k_c) mod M
    int32_t off;       // first coefficient of the band in a row
    int32_t fft;       // FftDesc index: length M, or P for Bluestein
    int32_t chirp;     // -1, or offset of exp(-i pi m^2 / M), m < M, in the chirp pool
    int32_t kern;      // offset of DFT_P(b)/P in the kernel pool (Bluestein only)
    int32_t n;         // transform length: M, or P for Bluestein
    float inv_M;
};

// One workgroup of a band kernel: band `band` for signals s0 .. s0 + count - 1,
// transformed as 2^lgnb interleaved sequences (count <= 2^lgnb). The band's
// record is repeated here, so a workgroup reads everything it needs to start
// its loads in one step.
struct WorkItem {
    int32_t band;
    int32_t s0;
    int32_t count;
    int32_t lgnb;
    int32_t fast;      // kItemFast* flags
    BandDev bd;
};

// Work item flags. A band kernel's fast load phases read entries up to
// kFastReach(M, st) = M - 1 + 3 st past the band's first one (st = threads per
// sequence) through affine addresses; the plan sets a flag only where every
// such read stays inside the data, the workspace guard or the table guard.
constexpr int32_t kItemFastRoute = 1;    // analysis router: 0 < k < L, Z and router tables
constexpr int32_t kItemFastCoef = 2;     // synthesis: coefficient reads stay inside the row set
// Guard, in complex entries, after the packed spectrum in the analysis
// workspace and after the per-coefficient tables.
constexpr int kFastGuard = 4096;

// A band whose transform (length M, or Bluestein P) exceeds one workgroup's
// LDS: it is transformed by a four-step FFT n = n1 * n2 through a per-signal
// global buffer (region hoff .. hoff + n of each signal's huge-band buffer).
struct BigDesc {
    int32_t band;
    int32_t n, n1, n2;
    int32_t fftn;            // FftDesc of n: its tables give omega_n for the four-step twiddles
    int32_t fft1, fft2;      // FftDescs of the column (n1) and row (n2) transforms
    int32_t lga, lgb;        // log2 of the columns / rows per workgroup
    int32_t hoff;
    int32_t pad;
};

// One workgroup of a huge-band pass: band big, signal sig, tile index tile.
struct BigItem {
    int32_t big;
    int32_t sig;
    int32_t tile;
    int32_t pad;
};

// Largest prime factor of n above 16 (the radix of a matrix-core stage), or 0.
inline int mfma_prime(int n) {
    int best = 0;
    for (int p = 2; p * p <= n; ++p)
        while (n % p == 0) {
            if (p > 16) best = p;
            n /= p;
        }
    return n > 16 && n > best ? n : best;
}

// LDS slots of nb = 2^lgnb interleaved sequences of length n (stride nb + 1),
// with room for a matrix-core stage's root table (entries 0..R): the unused
// slot of each row (plus one row when R = n), or R + 1 slots after a single
// sequence.
inline int lds_slots(int n, int lgnb) {
    const int R = mfma_prime(n);
    if (lgnb) return (R == n ? n + 1 : n) * ((1 << lgnb) + 1);
    return n + (R ? R + 1 : 0);
}

}  // namespace nsg
