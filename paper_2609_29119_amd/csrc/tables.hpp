// Device-visible table records shared by the host plan builder and the HIP
// kernels. Plain structs only: the host fills them in fp64 and stores fp32.
#pragma once

#include <cstdint>

namespace nsg {

// Largest prime handled by the direct odd-radix Stockham stage. Lengths with a
// larger prime factor are transformed with Bluestein's chirp-z algorithm over a
// 7-smooth length P >= 2M - 1.
constexpr int kGenericMaxRadix = 61;
constexpr int kMaxStages = 28;

// One transform length n: Stockham stages of the given radices, applied in
// order, and the offset of its twiddles omega_n^t = exp(-2 pi i t / n),
// t = 0..n-1, in the twiddle pool.
struct FftDesc {
    int32_t n;
    int32_t nstages;
    int32_t tw;
    int32_t max_generic;     // largest generic (odd prime >= 11) radix, 0 if none
    // two-level twiddles: omega_n^t = hi[t >> lg] * lo[t & (2^lg - 1)], with
    // hi at tw + n (ceil(n / 2^lg) values) and lo right after it (2^lg values)
    int32_t lg;
    int32_t nhi;
    int16_t radix[kMaxStages];
};

// LDS slots reserved for the two-level twiddles of any length up to 16384.
constexpr int kTwSlots = 288;
// LDS slots reserved for the table of a generic odd-prime radix.
constexpr int kWrSlots = 64;

// One band of the layout as the band kernels see it.
struct BandDev {
    int32_t k_lo;      // first support bin
    int32_t M;         // band length = support width
    int32_t rot;       // slot of bin k_lo: (k_lo - k_c) mod M
    int32_t off;       // first coefficient of the band in a row
    int32_t fft;       // FftDesc index: length M, or P for Bluestein
    int32_t chirp;     // -1, or offset of exp(-i pi m^2 / M), m < M, in the chirp pool
    int32_t kern;      // offset of DFT_P(b)/P in the kernel pool (Bluestein only)
    float inv_M;
};

// One workgroup of a band kernel: band `band` for signals s0 .. s0 + count - 1.
struct WorkItem {
    int32_t band;
    int32_t s0;
    int32_t count;
    int32_t pad;
};

// A band whose transform (length M, or Bluestein P) exceeds one workgroup's
// LDS: it is transformed by a four-step FFT n = n1 * n2 through a per-signal
// global buffer (region hoff .. hoff + n of each signal's huge-band buffer).
struct BigDesc {
    int32_t band;
    int32_t n, n1, n2;
    int32_t fftn;            // FftDesc of n: its tables give omega_n for the four-step twiddles
    int32_t fft1, fft2;      // FftDescs of the column (n1) and row (n2) transforms
    int32_t tile_a, tile_b;  // columns / rows per workgroup
    int32_t ld_a, ld_b;
    int32_t hoff;
};

// One workgroup of a huge-band pass: band big, signal sig, tile index tile.
struct BigItem {
    int32_t big;
    int32_t sig;
    int32_t tile;
    int32_t pad;
};

// LDS slots holding n complex values under the padded index i + i/8.
inline int lds_slots(int n) { return n + (n > 0 ? (n - 1) / 8 : 0) + 1; }

}  // namespace nsg
