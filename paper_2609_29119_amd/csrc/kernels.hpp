// HIP kernels of the packed constant-Q transform (Sec. 3, eqs. 5-10).
//
// Data layout in HBM (per signal, b signals back to back):
//   x      N float32                          input / output signal
//   Y      L complex64, row k1 of length L2  four-step intermediate
//   Z      L complex64, natural order         packed spectrum Z = F_L P x
//   c / W  C complex64, band offsets          coefficients / weighted band spectra
//
// Every kernel stages its sequences in LDS as 2^lgnb interleaved sequences
// (element i of sequence t at i*S + t, see fft_lds.hpp) and transforms them
// with lds_fft.
#pragma once

#include <hip/hip_runtime.h>

#include <type_traits>

#include "fft_lds.hpp"

namespace nsg {

// Ask for at least two waves per SIMD so LDS-bound stages can overlap; this
// caps each kernel at 256 VGPRs per lane.
#define NSG_OCC __attribute__((amdgpu_waves_per_eu(2)))
// The 256 x 8 and 64 x 8 band kernels gain from six waves per SIMD (at most
// 80 VGPRs, no spills); the larger tiers do not.
#define NSG_OCC_BAND __attribute__((amdgpu_waves_per_eu(((NT == 256 || NT == 64) && EPT == 8) ? 6 : 2)))

struct Tables {
    const BandDev* bands;
    const FftDesc* ffts;
    const float2* tw;        // twiddle pool
    const float2* omega;     // exp(-2 pi i k / N), k = 0..L
    const int32_t* owner;    // first band covering bin k | count << 24, k = 0..L
    const int32_t* bandbase; // off - k_lo per band
    const int4* gather;      // per bin k = 0..L: covering bands of k and of L - k (one or two int4)
    const float2* chirp;     // Bluestein exp(-i pi m^2 / M)
    const float2* kern;      // Bluestein DFT_P(b) / P
    const float2* tw4_hi;
    const float2* tw4_lo;
    const float* slicewin;
    const WorkItem* items;   // work items of the band kernels, all buckets
    const BigDesc* bigs;     // huge bands
    const BigItem* bigitems; // work items of the huge-band passes
};

struct Pass {
    int L1, L2;
    int lgnb;                // log2 of the columns (pass A) or rows (pass B) per workgroup
    int ntile;
    int fft;                 // FftDesc index of the pass length
    int ntw;                 // its stage-twiddle count
    int split;               // four-step twiddles: hi[t >> split] * lo[t & (2^split - 1)]
    int nhi4;                // number of hi values
    int L;
};

// Sliced input: slice s0 + sig of a signal x[n] with hop H, front pad H.
struct SliceIn {
    int enabled;
    int s0;
    long long n;
    int H;
};

// Hardware dispatches workgroup b to XCD b mod 8; give each XCD a contiguous
// range of logical ids so neighbouring tiles and bands share its L2.
__device__ __forceinline__ int xcd_remap(int b, int G) {
    const int x = b & 7, i = b >> 3;
    const int q = G >> 3, r = G & 7;
    return x * q + (x < r ? x : r) + i;
}

// Load phase shared by the kernels: thread tid takes the elements
// e = tid + j NT < total, U at a time. get(e) performs the element's global
// reads and touches only valid addresses for every 0 <= e < total (callers
// clamp indices and mask the value in put); put(e, v) consumes them. All U
// gets are issued before the first put, so a wave keeps U elements' reads in
// flight instead of waiting for each element in turn.
// Makes v's registers opaque: the loads producing v must complete here,
// so the compiler cannot sink them into the (conditional) consumer.
template <class V>
__device__ __forceinline__ void pin(V& v) {
    static_assert(sizeof(V) % 4 == 0, "pin expects 32-bit fields");
    uint32_t* w = reinterpret_cast<uint32_t*>(&v);
#pragma unroll
    for (int i = 0; i < static_cast<int>(sizeof(V) / 4); ++i) asm volatile("" : "+v"(w[i]));
}

template <int NT, int U, class Get, class Put>
__device__ __forceinline__ void load_phase(int total, Get get, Put put) {
    using V = decltype(get(0));
    for (int base = threadIdx.x; base < total; base += U * NT) {
        V v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = get(min(base + u * NT, total - 1));
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (base + u * NT < total) put(base + u * NT, v[u]);
    }
}

// LDS of the pass kernels: four-step twiddles (hi then lo, pass A only), data.
__device__ __forceinline__ void pass_lds(float2* lds, const Pass& p, bool with_tw4, float2*& t4, float2*& buf) {
    t4 = lds;
    buf = t4 + (with_tw4 ? p.nhi4 + (1 << p.split) : 0);
}

template <int NT>
__device__ __forceinline__ void load_tw4(float2* t4, const Pass& p, const Tables& T) {
    const int nlo = 1 << p.split;
    load_phase<NT, 2>(
        p.nhi4 + nlo, [&](int i) { return *(i < p.nhi4 ? T.tw4_hi + i : T.tw4_lo + (i - p.nhi4)); },
        [&](int i, float2 v) { t4[i] = v; });
}

// The same table in two steps, so that its global reads can overlap other
// reads: tw4_fetch issues the read of entry threadIdx.x into a register,
// tw4_store writes it to LDS later and reads the entries from NT on directly.
template <int NT>
__device__ __forceinline__ float2 tw4_fetch(const Pass& p, const Tables& T) {
    const int i = min(static_cast<int>(threadIdx.x), p.nhi4 + (1 << p.split) - 1);
    return *(i < p.nhi4 ? T.tw4_hi + i : T.tw4_lo + (i - p.nhi4));
}
template <int NT>
__device__ __forceinline__ void tw4_store(float2* t4, float2 v, const Pass& p, const Tables& T) {
    const int n = p.nhi4 + (1 << p.split);
    if (static_cast<int>(threadIdx.x) < n) t4[threadIdx.x] = v;
    load_phase<NT, 2>(
        n - NT,
        [&](int j) {
            const int i = j + NT;
            return *(i < p.nhi4 ? T.tw4_hi + i : T.tw4_lo + (i - p.nhi4));
        },
        [&](int j, float2 w) { t4[j + NT] = w; });
}

__device__ __forceinline__ float2 tw4(const float2* t4, const Pass& p, int t) {
    return cmul(t4[t >> p.split], t4[p.nhi4 + (t & ((1 << p.split) - 1))]);
}

// -------------------------------------------------- packed FFT, pass A (columns)
// Loads z_j = x_{2j} + i x_{2j+1} (eq. 5) for j = n1 L2 + n2 over a tile of
// columns n2, runs the length-L1 column DFTs, multiplies by omega_L^{n2 k1} and
// writes Y[k1 L2 + n2]. SLICED: z_j comes from slice s0 + sig of a long
// signal, windowed (Sec. 4). Persistent like pass B: the descriptor, stage
// twiddles and four-step twiddles sit in LDS, and the next tile's inputs are
// read into registers while the current tile is transformed.
template <int NT, int EPT, bool SLICED>
__global__ __launch_bounds__(NT) NSG_OCC void k_fwd_a(const float* __restrict__ x, float2* __restrict__ Y,
                                                      Pass p, Tables T, SliceIn sl, int batch, long long sig_stride) {
    extern __shared__ float2 lds[];
    __shared__ FftDesc fdl;
    const FftDesc* fd = T.ffts + p.fft;
    float2 *t4, *buf;
    pass_lds(lds, p, true, t4, buf);
    float2* twl = buf;
    buf += p.ntw;
    for (int i = threadIdx.x; i < static_cast<int>(sizeof(FftDesc) / 4); i += NT)
        reinterpret_cast<int*>(&fdl)[i] = reinterpret_cast<const int*>(fd)[i];
    for (int i = threadIdx.x; i < p.ntw; i += NT) twl[i] = T.tw[fd->stw + i];
    load_tw4<NT>(t4, p, T);
    const int G = p.ntile * batch;
    const int nbm = (1 << p.lgnb) - 1, S = seq_stride(p.lgnb);
    const int tot = p.L1 << p.lgnb;
    // per element: (x_2j, x_2j+1) or, sliced, the two samples and their window
    using Pre = typename std::conditional<SLICED, float4, float2>::type;
    Pre pre[EPT];
    // padded coordinate of sample 2j of slice s is s H + 2j; the signal
    // starts at padded H. Reads are clamped into the tile and the signal.
    auto fetch = [&](int t) {
        const int tile = t % p.ntile, sig = t / p.ntile;
        const int n2a = tile << p.lgnb;
        const int cmax = min(nbm + 1, p.L2 - n2a) - 1;
#pragma unroll
        for (int u = 0; u < EPT; ++u) {
            const int e = min(static_cast<int>(threadIdx.x) + u * NT, tot - 1);
            const int j = __mul24(e >> p.lgnb, p.L2) + n2a + min(e & nbm, cmax);
            if constexpr (SLICED) {
                const long long base = (long long)(sl.s0 + sig) * sl.H - sl.H;
                const long long tt = base + 2 * (long long)j;
                const long long last = sl.n - 1;
                const long long t0 = tt < 0 ? 0 : (tt > last ? last : tt);
                const long long t1 = tt + 1 < 0 ? 0 : (tt + 1 > last ? last : tt + 1);
                pre[u] = make_float4(x[t0], x[t1], T.slicewin[2 * j], T.slicewin[2 * j + 1]);
            } else {
                const float2* z = reinterpret_cast<const float2*>(x + (long long)sig * sig_stride);
                pre[u] = at32(z, j);
            }
        }
    };
    int t = blockIdx.x;
    if (t < G) fetch(t);
    for (; t < G; t += gridDim.x) {
        const int tile = t % p.ntile, sig = t / p.ntile;
        const int n2a = tile << p.lgnb;
        const int cols = min(nbm + 1, p.L2 - n2a);
#pragma unroll
        for (int u = 0; u < EPT; ++u) {
            const int e = threadIdx.x + u * NT;
            if (e < tot) {
                const int c = e & nbm, n1 = e >> p.lgnb;
                float2 v = make_float2(0.f, 0.f);
                if (c < cols) {
                    if constexpr (SLICED) {
                        const long long base = (long long)(sl.s0 + sig) * sl.H - sl.H;
                        const long long tt = base + 2 * (long long)(__mul24(n1, p.L2) + n2a + c);
                        if (tt >= 0 && tt < sl.n) v.x = pre[u].x * pre[u].z;
                        if (tt + 1 >= 0 && tt + 1 < sl.n) v.y = pre[u].y * pre[u].w;
                    } else {
                        v = pre[u];
                    }
                }
                buf[__mul24(n1, S) + c] = v;
            }
        }
        __syncthreads();
        if (t + static_cast<int>(gridDim.x) < G) fetch(t + gridDim.x);
        lds_fft<NT, EPT>(buf, S, p.lgnb, &fdl, T.tw, twl);
        float2* Ys = Y + (long long)sig * p.L;
        for (int e = threadIdx.x; e < tot; e += NT) {
            const int c = e & nbm, k1 = e >> p.lgnb;
            if (c < cols) {
                const int n2 = n2a + c;
                at32(Ys, __mul24(k1, p.L2) + n2) = cmul(buf[__mul24(k1, S) + c], tw4(t4, p, __mul24(n2, k1)));
            }
        }
        __syncthreads();
    }
}

__device__ __forceinline__ float4 make_float4_2(float2 a, float2 b) { return make_float4(a.x, a.y, b.x, b.y); }

// X_q = sum of the weighted band spectra W over the (at most three) bands
// covering bin q. The bin's half-record `head` holds the first band's W
// index with the count in bits 29..31, `steps` the int16 steps to the second
// and third bands' indices (0 where absent, so every index stays valid). All
// three reads are issued unconditionally.
__device__ __forceinline__ float2 gather_bin(const float2* __restrict__ Ws, int head, int steps) {
    const int i0 = head & ((1 << 29) - 1), cnt = static_cast<int>(static_cast<unsigned>(head) >> 29);
    const int i1 = i0 + static_cast<int>(static_cast<short>(steps & 0xFFFF));
    const int i2 = i1 + (steps >> 16);
    const float2 a = at32(Ws, i0), b = at32(Ws, i1), c = at32(Ws, i2);
    // masks instead of branches, so the compiler cannot sink the reads
    const float mb = cnt > 1 ? 1.f : 0.f, mc = cnt > 2 ? 1.f : 0.f;
    return make_float2(a.x + mb * b.x + mc * c.x, a.y + mb * b.y + mc * c.y);
}

// The same sum from a wide half-record: `head` as above, i1 and i2 the
// second and third bands' absolute W indices (the first's where absent).
__device__ __forceinline__ float2 gather_bin_abs(const float2* __restrict__ Ws, int head, int i1, int i2) {
    const int i0 = head & ((1 << 29) - 1), cnt = static_cast<int>(static_cast<unsigned>(head) >> 29);
    const float2 a = at32(Ws, i0), b = at32(Ws, i1), c = at32(Ws, i2);
    const float mb = cnt > 1 ? 1.f : 0.f, mc = cnt > 2 ? 1.f : 0.f;
    return make_float2(a.x + mb * b.x + mc * c.x, a.y + mb * b.y + mc * c.y);
}

// ------------------------------- inverse packed FFT, pass A, with overlap-add
// X_q for the packed bins of a tile is summed from the bands that cover the
// bin (no atomics: every packed bin is produced by exactly one thread), made
// real at DC and Nyquist, and retangled into
//   Z_q = (1/2)[(1 + i conj(w_q)) X_q + (1 - i conj(w_q)) conj(X_{L-q})]   (eq. 9).
// Bins pair up with their mirrors: for q = n1 L2 + n2 with 0 < n2 < L2,
// L - q = (L1 - 1 - n1) L2 + (L2 - n2). A tile holds H = 2^lgnb / 2 primary
// columns n2 in [0, L2/2] in slots 0..H-1 and their mirror columns L2 - n2
// in slots H..2H-1, so one thread gathers X_q and X_{L-q} once and emits both
// Z_q and Z_{L-q}. Columns equal to their mirror (0, and L2/2 for even L2)
// pair within the column and leave the mirror slot unused. With a single
// column per tile (lgnb = 0) tiles are plain columns. The inverse DFT is
// taken as conj(F_L conj(Z)) / L.
__device__ __forceinline__ float2 retangle_conj(float2 om, float2 xq, float2 xm) {
    const float2 pa = make_float2(1.f + om.y, om.x);      // 1 + i conj(w), om = (cos, -sin)
    const float2 pb = make_float2(1.f - om.y, -om.x);     // 1 - i conj(w)
    const float2 z = cadd(cmul(pa, xq), cmul(pb, conjf2(xm)));
    return make_float2(0.5f * z.x, -0.5f * z.y);          // conj(Z)
}

// WIDE: the plan's bin records are the 32-byte form (absolute indices).
template <int NT, int EPT, bool WIDE>
__global__ __launch_bounds__(NT) NSG_OCC void k_inv_a(const float2* __restrict__ W, float2* __restrict__ Y,
                                                      Pass p, Tables T, int batch, long long C) {
    extern __shared__ float2 lds[];
    float2 *t4, *buf;
    pass_lds(lds, p, true, t4, buf);
    // the four-step twiddles are needed only by the final store: their reads
    // go out first and land while the bin records are read
    const float2 t4pre = tw4_fetch<NT>(p, T);
    const int G = p.ntile * batch;
    const int lid = xcd_remap(blockIdx.x, G);
    const int tile = lid % p.ntile, sig = lid / p.ntile;
    const int nb = 1 << p.lgnb, S = seq_stride(p.lgnb);
    const bool pair = nb >= 2;
    const int lgH = pair ? p.lgnb - 1 : 0, H = 1 << lgH;
    const int c0 = tile << lgH;                                      // first primary column
    const int ncols = min(H, (pair ? (p.L2 >> 1) + 1 : p.L2) - c0);  // primary columns here
    const int tot = p.L1 << lgH;
    const float2* Ws = W + (long long)sig * C;
    // U elements at a time: the bin record (of q and L - q) and the twiddle of
    // q, then the W values it names, then the retangles; indices are clamped
    // into the tile
    constexpr int U = 4;
    for (int base = threadIdx.x; base < tot; base += U * NT) {
        int4 g[U], g2[U];
        float2 oq[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int e = min(base + u * NT, tot - 1);
            const int q = __mul24(e >> lgH, p.L2) + c0 + min(e & (H - 1), ncols - 1);
            if constexpr (WIDE) {
                g[u] = at32(T.gather, 2 * q);      // bins q and L - q
                g2[u] = at32(T.gather, 2 * q + 1);
            } else {
                g[u] = at32(T.gather, q);          // bins q and L - q
            }
            oq[u] = at32(T.omega, q);
        }
        float2 xq[U], xm[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if constexpr (WIDE) {
                xq[u] = gather_bin_abs(Ws, g[u].x, g[u].y, g[u].z);
                xm[u] = gather_bin_abs(Ws, g[u].w, g2[u].x, g2[u].y);
            } else {
                xq[u] = gather_bin(Ws, g[u].x, g[u].y);
                xm[u] = gather_bin(Ws, g[u].z, g[u].w);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int e = base + u * NT;
            const int c = e & (H - 1), n1 = e >> lgH;
            if (e < tot && c < ncols) {
                const int n2 = c0 + c;
                if (n1 == 0 && n2 == 0) { xq[u].y = 0.f; xm[u].y = 0.f; }    // DC and Nyquist
                buf[__mul24(n1, S) + c] = retangle_conj(oq[u], xq[u], xm[u]);
                // omega_N^{L-q} = -conj(omega_N^q), as omega_N^L = -1
                if (pair && n2 != 0 && 2 * n2 != p.L2)
                    buf[__mul24(p.L1 - 1 - n1, S) + H + c] =
                        retangle_conj(make_float2(-oq[u].x, oq[u].y), xm[u], xq[u]);
            }
        }
    }
    tw4_store<NT>(t4, t4pre, p, T);
    __syncthreads();
    lds_fft<NT, EPT>(buf, S, p.lgnb, T.ffts + p.fft, T.tw);
    __syncthreads();
    float2* Ys = Y + (long long)sig * p.L;
    // output column of a slot (primary or mirror), -1 for an unused slot
    auto column = [&](int slot) {
        const int c = slot & (H - 1), n2 = c0 + c;
        const bool mirror = pair && slot >= H;
        if (c >= ncols || (mirror && (n2 == 0 || 2 * n2 == p.L2))) return -1;
        return mirror ? p.L2 - n2 : n2;
    };
    for (int e = threadIdx.x; e < (p.L1 << p.lgnb); e += NT) {
        const int slot = e & (nb - 1), k1 = e >> p.lgnb;
        const int col = column(slot);
        if (col >= 0) at32(Ys, __mul24(k1, p.L2) + col) = cmul(buf[__mul24(k1, S) + slot], tw4(t4, p, __mul24(col, k1)));
    }
}

// ----------------------------------------------------- pass B (rows), both ways
// Row k1 of Y (length L2) is transformed; output k = k1 + L1 k2.
// INVERSE = false: Z[k] = result (natural order).
// INVERSE = true : z_k = conj(result) / L, unpacked to x_{2k}, x_{2k+1} (P^{-1}).
// Persistent: workgroup w takes tiles w, w + gridDim.x, ... (tile = 2^lgnb
// rows of one signal). The stage twiddles of length L2 sit in LDS, so the
// only global reads are the tiles': the next tile's rows are read into
// registers while the current tile is transformed.
template <int NT, int EPT, bool INVERSE>
__global__ __launch_bounds__(NT) NSG_OCC void k_pass_b(const float2* __restrict__ Y, float2* __restrict__ out,
                                                       Pass p, Tables T, int batch, long long out_stride,
                                                       float inv_L) {
    extern __shared__ float2 lds[];
    // the descriptor and stage twiddles are read from LDS inside the loop:
    // any global read there would have to wait for the prefetched rows first
    __shared__ FftDesc fdl;
    const FftDesc* fd = T.ffts + p.fft;
    float2* twl = lds;
    float2* buf = lds + p.ntw;
    for (int i = threadIdx.x; i < static_cast<int>(sizeof(FftDesc) / 4); i += NT)
        reinterpret_cast<int*>(&fdl)[i] = reinterpret_cast<const int*>(fd)[i];
    for (int i = threadIdx.x; i < p.ntw; i += NT) twl[i] = T.tw[fd->stw + i];
    const int G = p.ntile * batch;
    const int nbm = (1 << p.lgnb) - 1, S = seq_stride(p.lgnb);
    const int tot = p.L2 << p.lgnb;
    const Div dl2 = mkdiv(p.L2);
    float2 pre[EPT];
    // rows past the tile's last one are read clamped and stored as zeros
    auto fetch = [&](int t) {
        const int tile = t % p.ntile, sig = t / p.ntile;
        const int k1a = tile << p.lgnb;
        const int last = __mul24(min(nbm + 1, p.L1 - k1a), p.L2) - 1;
        const float2* Ys = Y + (long long)sig * p.L + (long long)k1a * p.L2;
#pragma unroll
        for (int u = 0; u < EPT; ++u) pre[u] = at32(Ys, min(static_cast<int>(threadIdx.x) + u * NT, last));
    };
    int t = blockIdx.x;
    if (t < G) fetch(t);
    for (; t < G; t += gridDim.x) {
        const int tile = t % p.ntile, sig = t / p.ntile;
        const int k1a = tile << p.lgnb;
        const int rows = min(nbm + 1, p.L1 - k1a);
#pragma unroll
        for (int u = 0; u < EPT; ++u) {
            const int e = threadIdx.x + u * NT;
            if (e < tot) {
                int n2;
                const int r = qdiv(e, dl2, n2);
                buf[__mul24(n2, S) + r] = r < rows ? pre[u] : make_float2(0.f, 0.f);
            }
        }
        __syncthreads();
        if (t + static_cast<int>(gridDim.x) < G) fetch(t + gridDim.x);
        lds_fft<NT, EPT>(buf, S, p.lgnb, &fdl, T.tw, twl);
        float2* os = out + (long long)sig * out_stride;
        for (int e = threadIdx.x; e < tot; e += NT) {
            const int r = e & nbm, k2 = e >> p.lgnb;
            if (r < rows) {
                const float2 v = buf[__mul24(k2, S) + r];
                at32(os, k1a + r + __mul24(p.L1, k2)) = INVERSE ? make_float2(v.x * inv_L, -v.y * inv_L) : v;
            }
        }
        __syncthreads();
    }
}

// ------------------------------------------------------------ band analysis
// Entries of nb = 2^lg interleaved sequences of length n: thread tid owns
// sequence tid & (nb - 1) and its entries i = (tid >> lg) + j (NT >> lg) < n,
// U at a time; as in load_phase, all U gets are issued before the first put,
// and get only sees valid indices.
template <int NT, int U, class Get, class Put>
__device__ __forceinline__ void seq_phase(int n, int lg, Get get, Put put) {
    const int step = NT >> lg;
    using V = decltype(get(0));
    for (int i0 = static_cast<int>(threadIdx.x) >> lg; i0 < n; i0 += U * step) {
        V v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = get(min(i0 + u * step, n - 1));
#pragma unroll
        for (int u = 0; u < U; ++u) pin(v[u]);
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (i0 + u * step < n) put(i0 + u * step, v[u]);
    }
}

// Two consecutive complex values at element idx of base (a 16-byte access;
// idx need not be even: global accesses only need dword alignment).
__device__ __forceinline__ float4 ld2c(const float2* base, uint32_t idx) {
    return *reinterpret_cast<const float4*>(reinterpret_cast<const char*>(base) + idx * 8u);
}
__device__ __forceinline__ void st2c(float2* base, uint32_t idx, float4 v) {
    *reinterpret_cast<float4*>(reinterpret_cast<char*>(base) + idx * 8u) = v;
}

// The router's value for one entry (eq. 7): conj(u) with
// u = (1/2) w (1 - i w_k) Z_a + (1/2) w (1 + i w_k) conj(Z_b), r holding the two
// factors. Every load form of the router goes through this one expression,
// so the result bits do not depend on which form a work item takes.
// Written as explicit fused multiply-adds, so the compiler cannot contract
// it differently in different places.
__device__ __forceinline__ float2 route_value(float4 r, float2 za, float2 zb) {
    const float ux = fmaf(r.x, za.x, fmaf(-r.y, za.y, fmaf(r.z, zb.x, r.w * zb.y)));
    const float uy = fmaf(r.x, za.y, fmaf(r.y, za.x, fmaf(-r.z, zb.y, r.w * zb.x)));
    return make_float2(ux, -uy);
}

// The transform descriptor of a band work item, copied to LDS in two steps:
// desc_fetch issues its global reads into registers, desc_store writes them
// to LDS. Between the two the kernel issues its router or coefficient reads,
// so the descriptor's round trip overlaps theirs instead of preceding them.
template <int NT>
struct DescCopy {
    static constexpr int kWords = static_cast<int>(sizeof(FftDesc) / 4);
    static constexpr int kPer = (kWords + NT - 1) / NT;
    int w[kPer];
    __device__ __forceinline__ void fetch(const FftDesc* d) {
        const int* src = reinterpret_cast<const int*>(d);
#pragma unroll
        for (int u = 0; u < kPer; ++u) w[u] = src[min(static_cast<int>(threadIdx.x) + u * NT, kWords - 1)];
    }
    __device__ __forceinline__ void store(FftDesc* l) const {
        int* dst = reinterpret_cast<int*>(l);
#pragma unroll
        for (int u = 0; u < kPer; ++u) {
            const int i = static_cast<int>(threadIdx.x) + u * NT;
            if (i < kWords) dst[i] = w[u];
        }
    }
};

// Bluestein's middle step on the LDS sequences: v <- conj(v K) for the
// transformed kernel K (entries 0 .. n-1), sequence sg of this thread.
template <int NT>
__device__ __forceinline__ void blu_middle(float2* buf, int n, int lg, int S, int sg, const float2* K) {
    seq_phase<NT, 4>(
        n, lg, [&](int i) { return at32(K, i); },
        [&](int i, float2 kv) {
            const int a = __mul24(i, S) + sg;
            buf[a] = conjf2(cmul(buf[a], kv));
        });
}

// One workgroup per work item (band, signals s0 .. s0 + count - 1, interleaved
// as 2^lgnb sequences). For entry i < W of the band (bin k = k_lo + i; slots
// of entries W <= i < M, past the support, hold zero) the router (eq. 7) forms
//   u = (1/2) w [(1 - i w_k) Z_{k mod L} + (1 + i w_k) conj(Z_{-k mod L})]
// with w the band's weight at k (g for T, the S^dagger weight for S^dagger),
// places conj(u) at slot (k - k_c) mod M in LDS, and the band's inverse DFT
// (eq. 2) is conj(F_M conj(u)) / M. Bands whose length has a prime factor
// above kMfmaMaxRadix (or for which it is cheaper) use Bluestein's algorithm: with ch_m = exp(-i pi m^2/M),
// F_M v = ch * conj(F_P conj(F_P(ch v) * K)) where K = F_P(b)/P and b the
// cyclic chirp exp(+i pi t^2/M), |t| < M.
template <int NT, int EPT>
__global__ __launch_bounds__(NT) NSG_OCC_BAND void k_band_analysis(const float2* __restrict__ Z, float2* __restrict__ coef,
                                                              const float4* __restrict__ rt, Tables T, int item0,
                                                              int nitems, int batch, int L, long long C) {
    extern __shared__ float2 lds[];
    const WorkItem it = T.items[item0 + blockIdx.x];
    const int g = min(it.count, batch - it.s0);
    if (g <= 0) return;
    const BandDev& bd = it.bd;
    // the descriptor goes to LDS (the stage loop then issues no global
    // descriptor reads); its read overlaps the router's
    __shared__ FftDesc fdl;
    DescCopy<NT> dsc;
    dsc.fetch(T.ffts + bd.fft);
    float2* buf = lds;
    const int M = bd.M, n = bd.n;
    const int lg = it.lgnb, nb = 1 << lg, S = seq_stride(lg);
    const bool blu = bd.chirp >= 0;
    // this thread's sequence; sequences past the item's count read signal 0
    // and hold zeros
    const int sg = threadIdx.x & (nb - 1);
    const bool live = sg < g;
    const float2* Zb = Z + (long long)it.s0 * L;
    const uint32_t zrow = static_cast<uint32_t>(live ? sg : 0) * static_cast<uint32_t>(L);
    const float2* chb = T.chirp + (blu ? bd.chirp : 0);   // entry 0 is valid in every table
    const float4* rb = rt + bd.off;
    // the chirp is read only by Bluestein bands (a uniform branch around
    // two instances of each phase)
    struct RouteIn { float2 za, zb, ch; float4 r; };
    auto route = [&](auto blu_t) {
        constexpr bool BLU = decltype(blu_t)::value;
        seq_phase<NT, 4>(
            M, lg,
            [&](int i) {
                int slot = i + bd.rot;
                if (slot >= M) slot -= M;
                // entries past the support read a valid bin; their factors are zero
                const int k = bd.k_lo + min(i, bd.W - 1);
                const int a = (k == L) ? 0 : k;
                const int bm = (a == 0) ? 0 : L - a;
                return RouteIn{at32(Zb, zrow + a), at32(Zb, zrow + bm),
                               BLU ? at32(chb, slot) : make_float2(1.f, 0.f), at32(rb, i)};
            },
            [&](int i, const RouteIn& r) {
                int slot = i + bd.rot;
                if (slot >= M) slot -= M;
                float2 v = make_float2(0.f, 0.f);
                if (live && i < bd.W) {
                    v = route_value(r.r, r.za, r.zb);
                    if (BLU) v = cmul(v, r.ch);
                }
                buf[__mul24(slot, S) + sg] = v;
            });
    };
    // The same for a band inside 0 < k < L whose reads past its last entry
    // stay inside the workspace and table guards (the plan's item flag). A
    // thread takes pairs of entries (i, i + 1), i = 2 (p0 + j st): one
    // 16-byte read of Z_k, Z_{k+1}, one of the mirror pair Z_{L-k-1},
    // Z_{L-k} and two of the router factors, all at addresses affine in j;
    // entries past M are read but not used. The slot of entry i advances
    // by 2 st modulo M.
    auto route_fast = [&](auto blu_t) {
        constexpr bool BLU = decltype(blu_t)::value;
        constexpr int RP = 2;                     // pairs per batch
        const int st = NT >> lg, p0 = static_cast<int>(threadIdx.x) >> lg;
        const int wl = live ? bd.W : 0;
        const int st2 = 2 * st;
        int slot = 2 * p0 + bd.rot;               // < 2 M whenever 2 p0 < M
        slot = slot >= M ? slot - M : slot;
        uint32_t zo = zrow + static_cast<uint32_t>(bd.k_lo + 2 * p0);
        uint32_t mo = zrow + static_cast<uint32_t>(L - bd.k_lo - 2 * p0 - 1);
        for (int ib = 2 * p0; ib < M; ib += RP * st2) {
            float4 za[RP], zb[RP], r0[RP], r1[RP];
            float2 c0[RP], c1[RP];
            int sl[RP];
#pragma unroll
            for (int u = 0; u < RP; ++u) {
                za[u] = ld2c(Zb + u * st2, zo);
                zb[u] = ld2c(Zb - u * st2, mo);
                r0[u] = at32(rb + u * st2, static_cast<uint32_t>(ib));
                r1[u] = at32(rb + u * st2 + 1, static_cast<uint32_t>(ib));
                sl[u] = slot;
                if (BLU) {
                    const int s1 = slot + 1 == M ? 0 : slot + 1;
                    c0[u] = at32(chb, static_cast<uint32_t>(slot));
                    c1[u] = at32(chb, static_cast<uint32_t>(s1));
                }
                const uint32_t nx = static_cast<uint32_t>(slot + st2);
                slot = static_cast<int>(min(nx, nx - static_cast<uint32_t>(M)));
            }
            zo += RP * st2;
            mo -= RP * st2;
#pragma unroll
            for (int u = 0; u < RP; ++u) {
                const int i = ib + u * st2;
                // entry i: Z_k = za.xy, Z_{L-k} = zb.zw; entry i + 1: za.zw, zb.xy
                float2 v0 = route_value(r0[u], make_float2(za[u].x, za[u].y), make_float2(zb[u].z, zb[u].w));
                float2 v1 = route_value(r1[u], make_float2(za[u].z, za[u].w), make_float2(zb[u].x, zb[u].y));
                if (BLU) {
                    v0 = cmul(v0, c0[u]);
                    v1 = cmul(v1, c1[u]);
                }
                if (i >= wl) v0 = make_float2(0.f, 0.f);
                if (i + 1 >= wl) v1 = make_float2(0.f, 0.f);
                const int s1 = sl[u] + 1 == M ? 0 : sl[u] + 1;
                if (i < M) buf[__mul24(sl[u], S) + sg] = v0;
                if (i + 1 < M) buf[__mul24(s1, S) + sg] = v1;
            }
        }
    };
    if (it.fast & kItemFastRoute) {
        if (blu) route_fast(std::true_type{});
        else route_fast(std::false_type{});
    } else {
        if (blu) route(std::true_type{});
        else route(std::false_type{});
    }
    dsc.store(&fdl);
    if (blu)
        for (int e = threadIdx.x; e < ((n - M) << lg); e += NT)
            buf[__mul24(M + (e >> lg), S) + (e & (nb - 1))] = make_float2(0.f, 0.f);
    __syncthreads();
    lds_fft<NT, EPT>(buf, S, lg, &fdl, T.tw);
    if (blu) {
        blu_middle<NT>(buf, n, lg, S, sg, T.kern + bd.kern);
        __syncthreads();
        lds_fft<NT, EPT>(buf, S, lg, &fdl, T.tw);
    }
    if (!live) return;
    float2* cb = coef + (long long)it.s0 * C + bd.off;
    const uint32_t crow = static_cast<uint32_t>(sg) * static_cast<uint32_t>(C);
    // mixed radix: c = conj(V) / M; Bluestein: c = conj(ch * conj(D)) / M = conj(ch) D / M
    if (blu) {
        seq_phase<NT, 4>(
            M, lg, [&](int i) { return at32(chb, i); },
            [&](int i, float2 chi) {
                at32(cb, crow + i) = cscale(cmul(conjf2(chi), buf[__mul24(i, S) + sg]), bd.inv_M);
            });
    } else {
        // pairs of entries (i, i + 1), i = 2 (p0 + j st), two at a time: one
        // 16-byte write per pair at addresses affine in j (scalar base, one
        // lane offset); a lone last entry is written on its own
        const int st = NT >> lg, p0 = static_cast<int>(threadIdx.x) >> lg;
        const int st2 = 2 * st, stS = __mul24(st2, S);
        int a = __mul24(2 * p0, S) + sg;
        for (int ib = 2 * p0; ib < M; ib += 2 * st2) {
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int i = ib + u * st2;
                if (i + 1 < M) {
                    const float2 v0 = buf[a + u * stS], v1 = buf[a + u * stS + S];
                    st2c(cb + u * st2, crow + static_cast<uint32_t>(ib),
                         make_float4(v0.x * bd.inv_M, -v0.y * bd.inv_M, v1.x * bd.inv_M, -v1.y * bd.inv_M));
                } else if (i < M) {
                    const float2 v0 = buf[a + u * stS];
                    at32(cb + u * st2, crow + static_cast<uint32_t>(ib)) = make_float2(v0.x * bd.inv_M, -v0.y * bd.inv_M);
                }
            }
            a += 2 * stS;
        }
    }
}

// ----------------------------------------------------------- band synthesis
// One workgroup per work item: U = F_M c (eq. 10), then the weighted band
// spectrum W[off + i] = w_i U[slot(k_lo + i)] in bin order for the support
// entries i < W (w = h for S, the T^dagger weight for T^dagger). Overlapping bands are summed later by the
// owner of each bin.
template <int NT, int EPT>
__global__ __launch_bounds__(NT) NSG_OCC_BAND void k_band_synthesis(const float2* __restrict__ coef, float2* __restrict__ W,
                                                               const float* __restrict__ wt, Tables T, int item0,
                                                               int nitems, int batch, long long C) {
    extern __shared__ float2 lds[];
    const WorkItem it = T.items[item0 + blockIdx.x];
    const int g = min(it.count, batch - it.s0);
    if (g <= 0) return;
    const BandDev& bd = it.bd;
    __shared__ FftDesc fdl;
    DescCopy<NT> dsc;
    dsc.fetch(T.ffts + bd.fft);
    float2* buf = lds;
    const int M = bd.M, n = bd.n;
    const int lg = it.lgnb, nb = 1 << lg, S = seq_stride(lg);
    const bool blu = bd.chirp >= 0;
    const int sg = threadIdx.x & (nb - 1);
    const bool live = sg < g;
    const float2* chb = T.chirp + (blu ? bd.chirp : 0);   // entry 0 is valid in every table
    const float2* cb = coef + (long long)it.s0 * C + bd.off;
    const uint32_t crow = static_cast<uint32_t>(live ? sg : 0) * static_cast<uint32_t>(C);
    // fast form (the plan's item flag: reads up to entry M + 2 st stay in the
    // row): pairs of entries (i, i + 1), i = 2 (p0 + j st), one 16-byte read
    // of the coefficients each (and of the chirp for Bluestein)
    auto load_fast = [&](auto blu_t) {
        constexpr bool BLU = decltype(blu_t)::value;
        const int st = NT >> lg, p0 = static_cast<int>(threadIdx.x) >> lg;
        const int st2 = 2 * st, stS = __mul24(st2, S);
        int a = __mul24(2 * p0, S) + sg;
        for (int ib = 2 * p0; ib < M; ib += 2 * st2) {
            float4 cv[2], hv[2];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                cv[u] = ld2c(cb + u * st2, crow + static_cast<uint32_t>(ib));
                if (BLU) hv[u] = ld2c(chb + u * st2, static_cast<uint32_t>(ib));
            }
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int i = ib + u * st2;
                float2 v0 = make_float2(cv[u].x, cv[u].y), v1 = make_float2(cv[u].z, cv[u].w);
                if (BLU) {
                    v0 = cmul(v0, make_float2(hv[u].x, hv[u].y));
                    v1 = cmul(v1, make_float2(hv[u].z, hv[u].w));
                }
                if (!live) v0 = v1 = make_float2(0.f, 0.f);
                if (i < M) buf[a + u * stS] = v0;
                if (i + 1 < M) buf[a + u * stS + S] = v1;
            }
            a += 2 * stS;
        }
    };
    if (it.fast & kItemFastCoef) {
        if (blu) load_fast(std::true_type{});
        else load_fast(std::false_type{});
    } else if (blu) {
        seq_phase<NT, 4>(
            M, lg, [&](int i) { return make_float4_2(at32(cb, crow + i), at32(chb, i)); },
            [&](int i, float4 r) {
                buf[__mul24(i, S) + sg] = live ? cmul(make_float2(r.x, r.y), make_float2(r.z, r.w))
                                               : make_float2(0.f, 0.f);
            });
    } else {
        seq_phase<NT, 4>(
            M, lg, [&](int i) { return at32(cb, crow + i); },
            [&](int i, float2 v) { buf[__mul24(i, S) + sg] = live ? v : make_float2(0.f, 0.f); });
    }
    dsc.store(&fdl);
    if (blu)
        for (int e = threadIdx.x; e < ((n - M) << lg); e += NT)
            buf[__mul24(M + (e >> lg), S) + (e & (nb - 1))] = make_float2(0.f, 0.f);
    __syncthreads();
    lds_fft<NT, EPT>(buf, S, lg, &fdl, T.tw);
    if (blu) {
        blu_middle<NT>(buf, n, lg, S, sg, T.kern + bd.kern);
        __syncthreads();
        lds_fft<NT, EPT>(buf, S, lg, &fdl, T.tw);
    }
    if (!live) return;
    const float* w = wt + bd.off;
    float2* Wb = W + (long long)it.s0 * C + bd.off;
    struct OutIn { float2 ch; float w; };
    auto weigh = [&](auto blu_t) {
        constexpr bool BLU = decltype(blu_t)::value;
        seq_phase<NT, 4>(
            bd.W, lg,
            [&](int i) {
                int slot = i + bd.rot;
                if (slot >= M) slot -= M;
                return OutIn{BLU ? at32(chb, slot) : make_float2(1.f, 0.f), at32(w, i)};
            },
            [&](int i, const OutIn& r) {
                int slot = i + bd.rot;
                if (slot >= M) slot -= M;
                float2 u = buf[__mul24(slot, S) + sg];
                if (BLU) u = cmul(r.ch, conjf2(u));
                at32(Wb, crow + i) = cscale(u, r.w);
            });
    };
    // pairs of support entries (i, i + 1), i = 2 (p0 + j st): one 8-byte read
    // of the weights and one 16-byte write of W per pair (the weight table's
    // guard covers the reads past the support)
    auto weigh_fast = [&](auto blu_t) {
        constexpr bool BLU = decltype(blu_t)::value;
        const int st = NT >> lg, p0 = static_cast<int>(threadIdx.x) >> lg;
        const int st2 = 2 * st, Wd = bd.W;
        int slot = 2 * p0 + bd.rot;               // < 2 M whenever 2 p0 < W
        slot = slot >= M ? slot - M : slot;
        for (int ib = 2 * p0; ib < Wd; ib += 2 * st2) {
            float2 wv[2], h0[2], h1[2];
            int sl[2];
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                wv[u] = *reinterpret_cast<const float2*>(w + u * st2 + ib);
                sl[u] = slot;
                if (BLU) {
                    h0[u] = at32(chb, static_cast<uint32_t>(slot));
                    h1[u] = at32(chb, static_cast<uint32_t>(slot + 1 == M ? 0 : slot + 1));
                }
                const uint32_t nx = static_cast<uint32_t>(slot + st2);
                slot = static_cast<int>(min(nx, nx - static_cast<uint32_t>(M)));
            }
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const int i = ib + u * st2;
                const int s1 = sl[u] + 1 == M ? 0 : sl[u] + 1;
                float2 u0 = buf[__mul24(sl[u], S) + sg], u1 = buf[__mul24(s1, S) + sg];
                if (BLU) {
                    u0 = cmul(h0[u], conjf2(u0));
                    u1 = cmul(h1[u], conjf2(u1));
                }
                u0 = cscale(u0, wv[u].x);
                u1 = cscale(u1, wv[u].y);
                if (i + 1 < Wd) st2c(Wb + u * st2, crow + static_cast<uint32_t>(ib), make_float4_2(u0, u1));
                else if (i < Wd) at32(Wb + u * st2, crow + static_cast<uint32_t>(ib)) = u0;
            }
        }
    };
    if (blu) weigh_fast(std::true_type{});
    else weigh_fast(std::false_type{});
}

// ------------------------------------------------------------ huge bands
// Bands whose transform exceeds one workgroup run the same router, band DFTs
// and weighting as k_band_analysis / k_band_synthesis, but transform through
// a four-step FFT n = n1 n2 in a per-signal global buffer: the column pass
// (k_big_a) builds its input on the fly, the row pass (k_big_b) finishes the
// output.

struct BigArgs {
    const float2* Z;        // analysis input, [b][L]
    const float2* cin;      // synthesis input, [b][C]
    float2* cout;           // analysis output, [b][C]
    float2* W;              // synthesis output (weighted band spectra), [b][C]
    float2* H1;             // four-step intermediate, [b][Hn]
    float2* H2;             // Bluestein first-FFT output, [b][Hn]
    const float4* rt;       // analysis: router factors of the op
    const float* wt;        // synthesis: per-coefficient weights of the op
    int L;
    long long C, Hn;
    int analysis;
};

constexpr int kBigInRoute = 0, kBigInCoef = 1, kBigInBlu2 = 2;

// Column pass: input element j of the length-n sequence, columns c0..c0+cols
// of the n1 x n2 view j = r n2 + c, length-n1 DFTs, twiddle omega_n^{c k1}.
template <int NT, int EPT>
__global__ __launch_bounds__(NT) NSG_OCC void k_big_a(BigArgs a, Tables T, int item0, int nitems, int batch,
                                                      int in_mode) {
    extern __shared__ float2 lds[];
    const BigItem it = T.bigitems[item0 + xcd_remap(blockIdx.x, nitems)];
    if (it.sig >= batch) return;
    const BigDesc bg = T.bigs[it.big];
    const BandDev bd = T.bands[bg.band];
    const FftDesc* fdn = T.ffts + bg.fftn;
    const FftDesc* fd1 = T.ffts + bg.fft1;
    float2* t4 = lds;
    const int nt4 = fdn->nhi + (1 << fdn->lg);
    float2* buf = t4 + nt4;
    for (int i = threadIdx.x; i < nt4; i += NT) t4[i] = T.tw[fdn->full + fdn->n + i];
    const TwL w4{t4, fdn->nhi, fdn->lg};
    const int M = bd.M;
    const bool blu = bd.chirp >= 0;
    const int lg = bg.lga, nbm = (1 << lg) - 1, S = seq_stride(lg);
    const int c0 = it.tile << lg;
    const int cols = min(nbm + 1, bg.n2 - c0);
    const int tot = bg.n1 << lg;
    const long long hbase = (long long)it.sig * a.Hn + bg.hoff;
    for (int e = threadIdx.x; e < tot; e += NT) {
        const int c = e & nbm, r = e >> lg;
        const int j = __mul24(r, bg.n2) + c0 + c;
        float2 v = make_float2(0.f, 0.f);
        if (c < cols) {
            if (in_mode == kBigInBlu2) {
                v = conjf2(cmul(a.H2[hbase + j], T.kern[bd.kern + j]));
            } else if (j < M) {
                if (in_mode == kBigInRoute) {
                    int i = j - bd.rot;
                    if (i < 0) i += M;
                    if (i < bd.W) {   // slots past the support hold zero
                        const int k = bd.k_lo + i;
                        const float2* Zs = a.Z + (long long)it.sig * a.L;
                        const int ka = (k == a.L) ? 0 : k;
                        const int kb = (ka == 0) ? 0 : a.L - ka;
                        const float2 za = Zs[ka], zb = Zs[kb];
                        const float4 r = a.rt[bd.off + i];             // router factors
                        v = route_value(r, za, zb);
                    }
                } else {
                    v = a.cin[(long long)it.sig * a.C + bd.off + j];
                }
                if (blu) v = cmul(v, T.chirp[bd.chirp + j]);
            }
        }
        buf[__mul24(r, S) + c] = v;
    }
    __syncthreads();
    lds_fft<NT, EPT>(buf, S, lg, fd1, T.tw);
    __syncthreads();
    float2* Y = a.H1 + hbase;
    for (int e = threadIdx.x; e < tot; e += NT) {
        const int c = e & nbm, k1 = e >> lg;
        if (c < cols)
            Y[__mul24(k1, bg.n2) + c0 + c] = cmul(buf[__mul24(k1, S) + c], tw_at(w4, __mul24(c0 + c, k1)));
    }
}

// Row pass: rows r0..r0+rows of the intermediate, length-n2 DFTs, output
// k = k1 + n1 k2. second == 0: a Bluestein band's first FFT goes to H2, any
// other band finishes; second == 1: the Bluestein band finishes.
template <int NT, int EPT>
__global__ __launch_bounds__(NT) NSG_OCC void k_big_b(BigArgs a, Tables T, int item0, int nitems, int batch,
                                                      int second) {
    extern __shared__ float2 lds[];
    const BigItem it = T.bigitems[item0 + xcd_remap(blockIdx.x, nitems)];
    if (it.sig >= batch) return;
    const BigDesc bg = T.bigs[it.big];
    const BandDev bd = T.bands[bg.band];
    const FftDesc* fd2 = T.ffts + bg.fft2;
    float2* buf = lds;
    const int M = bd.M;
    const bool blu = bd.chirp >= 0;
    const int lg = bg.lgb, nbm = (1 << lg) - 1, S = seq_stride(lg);
    const int r0 = it.tile << lg;
    const int rows = min(nbm + 1, bg.n1 - r0);
    const int tot = bg.n2 << lg;
    const Div dn2 = mkdiv(bg.n2);
    const long long hbase = (long long)it.sig * a.Hn + bg.hoff;
    const float2* Y = a.H1 + hbase + (long long)r0 * bg.n2;
    for (int e = threadIdx.x; e < tot; e += NT) {
        int c;
        const int r = qdiv(e, dn2, c);
        buf[__mul24(c, S) + r] = r < rows ? Y[e] : make_float2(0.f, 0.f);
    }
    __syncthreads();
    lds_fft<NT, EPT>(buf, S, lg, fd2, T.tw);
    const bool to_mid = blu && !second;
    for (int e = threadIdx.x; e < tot; e += NT) {
        const int r = e & nbm, k2 = e >> lg;
        if (r >= rows) continue;
        const int k = r0 + r + __mul24(bg.n1, k2);
        const float2 v = buf[__mul24(k2, S) + r];
        if (to_mid) {
            a.H2[hbase + k] = v;
        } else if (k < M) {
            if (a.analysis) {
                // mixed radix: c = conj(V) / M; Bluestein: c = conj(ch) D / M
                const float2 o = blu ? cmul(conjf2(T.chirp[bd.chirp + k]), v) : conjf2(v);
                a.cout[(long long)it.sig * a.C + bd.off + k] = cscale(o, bd.inv_M);
            } else {
                const float2 u = blu ? cmul(T.chirp[bd.chirp + k], conjf2(v)) : v;
                int i = k - bd.rot;
                if (i < 0) i += M;
                if (i < bd.W) a.W[(long long)it.sig * a.C + bd.off + i] = cscale(u, a.wt[bd.off + i]);
            }
        }
    }
}

// ------------------------------------------------------ sliced overlap-add
// Output sample at padded position pp in [s0 H, (s0 + cnt) H) and inside the
// signal: the slice sb = pp / H starting there and the slice sb - 1 ending
// there contribute; slice s0 - 1 comes from the carry buffer (its upper half).
// Also saves the upper half of the chunk's last slice for the next chunk.
__global__ void k_ola(const float* __restrict__ y, const float* __restrict__ carry_in,
                      float* __restrict__ carry_out, float* __restrict__ xo, int s0, int cnt, int Ns,
                      long long n) {
    const int H = Ns / 2;
    const long long span = (long long)cnt * H;
    for (long long e = (long long)blockIdx.x * blockDim.x + threadIdx.x; e < span;
         e += (long long)gridDim.x * blockDim.x) {
        const long long pp = (long long)s0 * H + e;
        const long long t = pp - H;
        if (t >= 0 && t < n) {
            const int sb = (int)(pp / H);
            const int lb = (int)(pp - (long long)sb * H);    // local index in slice sb, in [0, H)
            float v = y[(long long)(sb - s0) * Ns + lb];
            const int sa = sb - 1;
            if (sa >= s0) v += y[(long long)(sa - s0) * Ns + lb + H];
            else if (sa >= 0) v += carry_in[lb];
            xo[t] = v;
        }
        if (e < H) carry_out[e] = y[(long long)(cnt - 1) * Ns + H + e];
    }
}

}  // namespace nsg
