// In-LDS mixed-radix Stockham FFT for one workgroup (gfx950, wave64).
//
// A workgroup of NT threads transforms nb = 2^lgnb sequences of length n in
// place. Element i of sequence t lives at LDS slot i*S + t with S = nb + 1
// (S = 1 for a single sequence): lanes that handle the same butterfly of
// neighbouring sequences touch neighbouring slots, and the odd stride keeps
// strided walks across the banks, so no padding or swizzle is needed.
//
// Each stage with radix R reads every butterfly's R inputs into registers,
// multiplies them by the stage twiddles, applies a compile-time length-R DFT
// and, after a barrier, writes the outputs in autosort order. The stage
// twiddles omega_{Ns R}^{r k} are precomputed per transform length, R - 1
// consecutive values per k, so a butterfly reads them with immediate offsets.
// The caller guarantees nb * n <= NT * EPT.
//
// All transforms are forward DFTs (eq. 1, exp(-2 pi i k j / n)); inverse
// transforms are obtained by conjugating input and output.
#pragma once

#include <hip/hip_runtime.h>

#include "radix_consts.hpp"
#include "tables.hpp"

namespace nsg {

__device__ __forceinline__ float2 cmul(float2 a, float2 b) {
    return make_float2(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}
__device__ __forceinline__ float2 cadd(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float2 csub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }
__device__ __forceinline__ float2 conjf2(float2 a) { return make_float2(a.x, -a.y); }
__device__ __forceinline__ float2 cscale(float2 a, float s) { return make_float2(a.x * s, a.y * s); }
// multiply by -i
__device__ __forceinline__ float2 mul_mi(float2 a) { return make_float2(a.y, -a.x); }

// ------------------------------------------------------------------ helpers

// The thread index made opaque to the optimiser. Each stage derives its
// indices from a fresh copy, so values of different stage kinds are not
// hoisted out of the stage loop and kept live together (which otherwise
// doubles the register footprint).
__device__ __forceinline__ int stage_tid() {
    int t = threadIdx.x;
    asm volatile("" : "+v"(t));
    return t;
}

// Exact quotient and remainder of 0 <= x < 2^22 by 0 < d < 2^22 through the
// fp32 reciprocal r = RN(1/d), with no correction step and no branch: the
// product p = RN((x + 1/2) r) (x + 1/2 is exact in fp32) is within a relative
// 2^-23 of y = (x + 1/2) / d, i.e. within (x + 1/2) 2^-23 / d < 1 / (2d),
// while y lies at least 1 / (2d) from every integer; so trunc(p) = floor(x/d).
struct Div {
    float r;
    int d;
};
// r = 1.0f / d: fp32 division is correctly rounded, so r = RN(1/d).
__device__ __forceinline__ Div mkdiv(int d) { return Div{1.0f / static_cast<float>(d), d}; }
// The same from a reciprocal the plan rounded once to fp32 (FftDesc).
__device__ __forceinline__ Div mkdiv(int d, float r) { return Div{r, d}; }
__device__ __forceinline__ int qdiv(int x, Div v, int& rem) {
    const int q = static_cast<int>((static_cast<float>(x) + 0.5f) * v.r);
    rem = x - __mul24(q, v.d);
    return q;
}

// Two-level table omega_n^t = hi[t >> lg] * lo[t & (2^lg - 1)] (four-step
// twiddles): hi values at t[0 .. nhi), lo values at t[nhi .. nhi + 2^lg).
struct TwL {
    const float2* t;
    int nhi;
    int lg;
};
__device__ __forceinline__ float2 tw_at(const TwL& w, int t) {
    return cmul(w.t[t >> w.lg], w.t[w.nhi + (t & ((1 << w.lg) - 1))]);
}

// Element idx of base through a 32-bit byte offset. With base uniform across
// the wave this is the scalar-base + vector-offset address form, which saves
// the 64-bit address arithmetic per access. The plan keeps every offset used
// this way below 2^32 bytes.
template <class T>
__device__ __forceinline__ const T& at32(const T* base, uint32_t idx) {
    return *reinterpret_cast<const T*>(reinterpret_cast<const char*>(base) + idx * static_cast<uint32_t>(sizeof(T)));
}
template <class T>
__device__ __forceinline__ T& at32(T* base, uint32_t idx) {
    return *reinterpret_cast<T*>(reinterpret_cast<char*>(base) + idx * static_cast<uint32_t>(sizeof(T)));
}

// ---------------------------------------------------------------- butterflies
// Forward DFTs of length R on v[0..R-1], in registers.

template <int R> struct Dft;

template <> struct Dft<2> {
    __device__ __forceinline__ static void run(float2* v) {
        const float2 a = v[0], b = v[1];
        v[0] = cadd(a, b);
        v[1] = csub(a, b);
    }
};

template <> struct Dft<4> {
    __device__ __forceinline__ static void run(float2* v) {
        const float2 t0 = cadd(v[0], v[2]), t1 = csub(v[0], v[2]);
        const float2 t2 = cadd(v[1], v[3]), t3 = mul_mi(csub(v[1], v[3]));
        v[0] = cadd(t0, t2);
        v[2] = csub(t0, t2);
        v[1] = cadd(t1, t3);
        v[3] = csub(t1, t3);
    }
};

template <> struct Dft<8> {
    __device__ __forceinline__ static void run(float2* v) {
        constexpr float r = 0.7071067811865475244008f;
        float2 e[4] = {v[0], v[2], v[4], v[6]};
        float2 o[4] = {v[1], v[3], v[5], v[7]};
        Dft<4>::run(e);
        Dft<4>::run(o);
        // o[q] *= exp(-2 pi i q / 8)
        const float2 o1 = make_float2(r * (o[1].x + o[1].y), r * (o[1].y - o[1].x));
        const float2 o2 = mul_mi(o[2]);
        const float2 o3 = make_float2(r * (o[3].y - o[3].x), -r * (o[3].x + o[3].y));
        v[0] = cadd(e[0], o[0]); v[4] = csub(e[0], o[0]);
        v[1] = cadd(e[1], o1);   v[5] = csub(e[1], o1);
        v[2] = cadd(e[2], o2);   v[6] = csub(e[2], o2);
        v[3] = cadd(e[3], o3);   v[7] = csub(e[3], o3);
    }
};

// Odd prime R: pair outputs q and R-q. With s_r = v_r + v_{R-r} and
// d_r = v_r - v_{R-r},
//   X_q     = v_0 + sum_r s_r cos(2 pi r q/R) - i sum_r d_r sin(2 pi r q/R)
//   X_{R-q} = v_0 + sum_r s_r cos(2 pi r q/R) + i sum_r d_r sin(2 pi r q/R).
template <int R> struct DftPrime {
    __device__ __forceinline__ static void run(float2* v) {
        constexpr int h = (R - 1) / 2;
        float2 s[h + 1], d[h + 1];
#pragma unroll
        for (int r = 1; r <= h; ++r) {
            s[r] = cadd(v[r], v[R - r]);
            d[r] = csub(v[r], v[R - r]);
        }
        const float2 v0 = v[0];
        float2 x0 = v0;
#pragma unroll
        for (int r = 1; r <= h; ++r) x0 = cadd(x0, s[r]);
#pragma unroll
        for (int q = 1; q <= h; ++q) {
            float2 A = v0, B = make_float2(0.f, 0.f);
#pragma unroll
            for (int r = 1; r <= h; ++r) {
                const float c = RootR<R>::re(r * q);
                const float sn = -RootR<R>::im(r * q);
                A.x += s[r].x * c; A.y += s[r].y * c;
                B.x += d[r].x * sn; B.y += d[r].y * sn;
            }
            v[q] = make_float2(A.x + B.y, A.y - B.x);       // A - i B
            v[R - q] = make_float2(A.x - B.y, A.y + B.x);   // A + i B
        }
        v[0] = x0;
    }
};

// R = A B by one Cooley-Tukey step in registers: input r = A b + a, output
// q = q1 + B q2; B-point DFTs over b, twiddles omega_R^{a q1}, A-point DFTs
// over a.
template <int A, int B> struct DftComposite {
    __device__ __forceinline__ static void run(float2* v) {
        constexpr int R = A * B;
        float2 y[A][B];
#pragma unroll
        for (int a = 0; a < A; ++a)
#pragma unroll
            for (int b = 0; b < B; ++b) y[a][b] = v[A * b + a];
#pragma unroll
        for (int a = 0; a < A; ++a) Dft<B>::run(y[a]);
#pragma unroll
        for (int a = 1; a < A; ++a)
#pragma unroll
            for (int q1 = 1; q1 < B; ++q1)
                y[a][q1] = cmul(y[a][q1], make_float2(RootR<R>::re(a * q1), RootR<R>::im(a * q1)));
#pragma unroll
        for (int q1 = 0; q1 < B; ++q1) {
            float2 z[A];
#pragma unroll
            for (int a = 0; a < A; ++a) z[a] = y[a][q1];
            Dft<A>::run(z);
#pragma unroll
            for (int q2 = 0; q2 < A; ++q2) v[q1 + B * q2] = z[q2];
        }
    }
};

template <> struct Dft<3> { __device__ __forceinline__ static void run(float2* v) { DftPrime<3>::run(v); } };
template <> struct Dft<5> { __device__ __forceinline__ static void run(float2* v) { DftPrime<5>::run(v); } };
template <> struct Dft<7> { __device__ __forceinline__ static void run(float2* v) { DftPrime<7>::run(v); } };
template <> struct Dft<11> { __device__ __forceinline__ static void run(float2* v) { DftPrime<11>::run(v); } };
template <> struct Dft<13> { __device__ __forceinline__ static void run(float2* v) { DftPrime<13>::run(v); } };
template <> struct Dft<6> { __device__ __forceinline__ static void run(float2* v) { DftComposite<2, 3>::run(v); } };
template <> struct Dft<9> { __device__ __forceinline__ static void run(float2* v) { DftComposite<3, 3>::run(v); } };
template <> struct Dft<10> { __device__ __forceinline__ static void run(float2* v) { DftComposite<2, 5>::run(v); } };
template <> struct Dft<12> { __device__ __forceinline__ static void run(float2* v) { DftComposite<3, 4>::run(v); } };
template <> struct Dft<14> { __device__ __forceinline__ static void run(float2* v) { DftComposite<2, 7>::run(v); } };
template <> struct Dft<15> { __device__ __forceinline__ static void run(float2* v) { DftComposite<3, 5>::run(v); } };
template <> struct Dft<16> { __device__ __forceinline__ static void run(float2* v) { DftComposite<4, 4>::run(v); } };

// -------------------------------------------------------------------- stages

// Stockham stage with compile-time radix R over nb = 2^lgnb sequences.
// Butterfly jj of sequence t reads in[jj + r m] (m = n/R), multiplies input r
// by omega_{Ns R}^{r k} (k = jj mod Ns, table tws[k (R-1) + r - 1]), applies
// the length-R DFT, and after a barrier writes out[(jj - k) R + k + r Ns].
// The twiddles omega_{Ns R}^{r k} come precomputed per stage (tws).
template <int R, int NT, int EPT>
__device__ __forceinline__ void stage_fixed(float2* buf, int n, int S, int lgnb, int Ns, float rns,
                                            const float2* __restrict__ tws) {
    constexpr int BPT = (EPT + R - 1) / R;
    const int tid = stage_tid();
    const int m = n / R;
    const int total = m << lgnb;
    const int nbm = (1 << lgnb) - 1;
    const int mS = __mul24(m, S), NsS = __mul24(Ns, S);
    const Div dns = mkdiv(Ns, rns);
    float2 v[BPT][R];
    int ob[BPT];
#pragma unroll
    for (int b = 0; b < BPT; ++b) {
        const int j = tid + b * NT;
        ob[b] = -1;
        if (j < total) {
            const int t = j & nbm, jj = j >> lgnb;
            int k = 0;
            if (Ns > 1) qdiv(jj, dns, k);
            int a = __mul24(jj, S) + t;
#pragma unroll
            for (int r = 0; r < R; ++r) {
                v[b][r] = buf[a];
                a += mS;
            }
            if (Ns > 1) {
                const float2* w = tws + __mul24(k, R - 1);
#pragma unroll
                for (int r = 1; r < R; ++r) v[b][r] = cmul(v[b][r], w[r - 1]);
            }
            Dft<R>::run(v[b]);
            ob[b] = __mul24(__mul24(jj - k, R) + k, S) + t;
        }
    }
    __syncthreads();
#pragma unroll
    for (int b = 0; b < BPT; ++b) {
        if (ob[b] >= 0) {
            int a = ob[b];
#pragma unroll
            for (int r = 0; r < R; ++r) {
                buf[a] = v[b][r];
                a += NsS;
            }
        }
    }
    __syncthreads();
}

// First half of a Stockham stage of odd prime radix R: each pair of inputs
// (r, R - r), r = 1..h, of every butterfly is multiplied by its stage twiddle
// and replaced in place by s_r = y_r + y_{R-r} (at r) and d_r = y_r - y_{R-r}
// (at R - r). Input 0 carries no twiddle.
template <int NT>
__device__ __forceinline__ void prime_fold(float2* buf, int n, int S, int lgnb, int Ns, int R, float rns,
                                           float rh, const float2* __restrict__ tws) {
    const int tid = stage_tid();
    const int m = n / R;
    const int h = (R - 1) >> 1;
    const int nbm = (1 << lgnb) - 1;
    const int mS = __mul24(m, S);
    const int totb = m << lgnb;
    const Div dns = mkdiv(Ns, rns), dh = mkdiv(h, rh);
    const int total = __mul24(totb, h);
    // four pairs at a time, all twiddle reads issued first
    constexpr int U = 4;
    for (int e0 = tid; e0 < total; e0 += U * NT) {
        int ia[U], ic[U];
        float2 wa[U], wc[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            int r1;
            const int j = qdiv(min(e0 + u * NT, total - 1), dh, r1);
            const int r = r1 + 1;
            const int jj = j >> lgnb;
            const int a0 = __mul24(jj, S) + (j & nbm);
            ia[u] = a0 + __mul24(r, mS);
            ic[u] = a0 + __mul24(R - r, mS);
            wa[u] = make_float2(1.f, 0.f);
            wc[u] = make_float2(1.f, 0.f);
            if (Ns > 1) {
                int k;
                qdiv(jj, dns, k);
                const int w0 = __mul24(k, R - 1) - 1;
                wa[u] = at32(tws, w0 + r);
                wc[u] = at32(tws, w0 + R - r);
            }
        }
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (e0 + u * NT < total) {
                const float2 ya = cmul(buf[ia[u]], wa[u]), yc = cmul(buf[ic[u]], wc[u]);
                buf[ia[u]] = cadd(ya, yc);
                buf[ic[u]] = csub(ya, yc);
            }
        }
    }
}

typedef float f32x4 __attribute__((ext_vector_type(4)));

// LDS slot of entry j of a prime stage's root table: the interleave's unused
// slot in row j (t = nb) for several sequences, or past the data for one.
// Entries j = 0..R are used (R <= n); the plan sizes the LDS accordingly.
__device__ __forceinline__ int root_slot0(int n, int S, int lgnb) { return lgnb ? (1 << lgnb) : n; }
__device__ __forceinline__ int root_step(int S, int lgnb) { return lgnb ? S : 1; }

// Stockham stage for an odd prime radix R (17 <= R <= kMfmaMaxRadix) known
// only at run time, on the matrix cores. After the fold, the outputs of butterfly column c are
//   X_q     = y_0 + A_q - i B_q,   X_{R-q} = y_0 + A_q + i B_q,   q = 0..h,
//   A_q = sum_r cos(2 pi q r / R) s_r,   B_q = sum_r sin(2 pi q r / R) d_r,
// i.e. products of fixed real h x h matrices with the real and imaginary
// parts of s and d. Real columns come in pairs (re, im) of one butterfly; the
// sine product reads d with the parts swapped, so the lane of each real part
// ends up with everything its two outputs need:
//   re lane: X_q = y0 + A_re + B_im,   X_{R-q} = y0 + A_re - B_im
//   im lane: X_q = y0 + A_im - B_re,   X_{R-q} = y0 + A_im + B_re.
// v_mfma_f32_16x16x4f32 operands: A (16 x 4) lane l row l % 16, column l / 16;
// B (4 x 16) lane l row l / 16, column l % 16; result (16 x 16) lane l, entry v
// at row 4 (l / 16) + v, column l % 16. The matrix entries come from the
// root table omega_R^j = (cos 2 pi j / R, -sin 2 pi j / R), j < R, which the
// stage copies into LDS (from the length's full root table, stride n / R)
// while the fold runs: entry (q, r) is omega_R^{q r mod R}, and each lane
// advances its exponent by 4 q mod R per column block of 4. Entry R holds
// zero; rows q > h and columns r > h read it. Each wave takes result tiles
// (column block, row block) round-robin and keeps at most kMfmaTilesPerWave of
// them until every wave has read its inputs; the caller guarantees
// mfma_tiles(totb, R) <= kMfmaTilesPerWave * NT / 64.
template <int NT>
__device__ __forceinline__ void stage_prime_mfma(float2* buf, int n, int S, int lgnb, int Ns, int R, float rns,
                                                 float rh, const float2* __restrict__ tws,
                                                 const float2* __restrict__ roots) {
    constexpr int NW = NT / 64;
    constexpr int TPW = kMfmaTilesPerWave;
    prime_fold<NT>(buf, n, S, lgnb, Ns, R, rns, rh, tws);
    const int tid = stage_tid();
    const int ts = root_step(S, lgnb);
    float2* tab = buf + root_slot0(n, S, lgnb);
    {
        const int stride = n / R;
        for (int j = tid; j <= R; j += NT)
            tab[__mul24(j, ts)] = j < R ? at32(roots, static_cast<uint32_t>(__mul24(j, stride))) : make_float2(0.f, 0.f);
    }
    __syncthreads();
    const int lane = tid & 63, wave = tid >> 6;
    const int m = n / R;
    const int h = (R - 1) >> 1;
    const int nbm = (1 << lgnb) - 1;
    const int mS = __mul24(m, S), NsS = __mul24(Ns, S);
    const int totb = m << lgnb;
    const int Qb = (h + 16) >> 4, Kb = (h + 3) >> 2;
    const int ntiles = ((totb + 7) >> 3) * Qb;
    // tile = cb Qb + qb with tile < 2^12 and Qb <= 17: (tile + 1/2) / Qb is at
    // least 1/34 from an integer, far beyond the reciprocal's error
    const float rqb = __builtin_amdgcn_rcpf(static_cast<float>(Qb));
    const int kk = lane >> 4, part = lane & 1;
    const int Rts = __mul24(R, ts);
    float* fb = reinterpret_cast<float*>(buf);
    f32x4 dc[TPW], ds[TPW];
    float y0[TPW];
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
        const int tile = wave + i * NW;            // wave-uniform
        dc[i] = f32x4{0.f, 0.f, 0.f, 0.f};
        ds[i] = f32x4{0.f, 0.f, 0.f, 0.f};
        y0[i] = 0.f;
        if (tile < ntiles) {
            const int cb = static_cast<int>((static_cast<float>(tile) + 0.5f) * rqb), qb = tile - cb * Qb;
            const int c = min((cb << 3) + ((lane & 15) >> 1), totb - 1);
            const int a0 = __mul24(c >> lgnb, S) + (c & nbm);
            // s_r.part at input r, d_r.(1 - part) at input R - r (r = 4 kb + kk + 1;
            // columns past h read inputs that the zero table entry cancels)
            int as = 2 * (a0 + __mul24(kk + 1, mS)) + part;
            int ad = 2 * (a0 + __mul24(R - kk - 1, mS)) + 1 - part;
            const int step = 8 * mS;
            // table exponent of entry (q, r) as a slot offset, and its step per
            // column block; rows past h sit on the zero entry (step R keeps them there)
            const int q = (qb << 4) + (lane & 15);
            int t, inc;
            if (q <= h) {
                t = __mul24(q, kk + 1);          // < 2 R
                t = t >= R ? t - R : t;
                inc = 4 * q;                      // < 2 R
                inc = inc >= R ? inc - R : inc;
                t = __mul24(t, ts);
                inc = __mul24(inc, ts);
            } else {
                t = Rts;
                inc = Rts;
            }
            // all blocks but the last: every column r <= h; two blocks at a
            // time, their LDS reads issued before the products
            int kb = 0;
            for (; kb + 2 < Kb; kb += 2) {
                float2 w[2];
                float sv[2], dv[2];
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    w[u] = tab[t];
                    sv[u] = fb[as + u * step];
                    dv[u] = fb[ad - u * step];
                    const uint32_t nx = static_cast<uint32_t>(t + inc);
                    t = static_cast<int>(min(nx, nx - static_cast<uint32_t>(Rts)));
                }
#pragma unroll
                for (int u = 0; u < 2; ++u) {
                    dc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(w[u].x, sv[u], dc[i], 0, 0, 0);
                    ds[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(w[u].y, dv[u], ds[i], 0, 0, 0);
                }
                as += 2 * step;
                ad -= 2 * step;
            }
            for (; kb < Kb; ++kb) {
                // in the last block, columns r = 4 kb + kk + 1 > h read the zero entry
                const int tu = (kb == Kb - 1 && 4 * kb + kk + 1 > h) ? Rts : t;
                const float2 w = tab[tu];
                const float sv = fb[as], dv = fb[ad];
                dc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(w.x, sv, dc[i], 0, 0, 0);
                ds[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(w.y, dv, ds[i], 0, 0, 0);
                as += step;
                ad -= step;
                const uint32_t nx = static_cast<uint32_t>(t + inc);
                t = static_cast<int>(min(nx, nx - static_cast<uint32_t>(Rts)));
            }
            y0[i] = fb[2 * a0 + part];
        }
    }
    __syncthreads();
    const Div dns = mkdiv(Ns, rns);
#pragma unroll
    for (int i = 0; i < TPW; ++i) {
        const int tile = wave + i * NW;
        if (tile < ntiles) {
            const int cb = static_cast<int>((static_cast<float>(tile) + 0.5f) * rqb), qb = tile - cb * Qb;
            const int c = (cb << 3) + ((lane & 15) >> 1);
            if (c < totb) {
                const int t = c & nbm, jj = c >> lgnb;
                int k = 0;
                if (Ns > 1) qdiv(jj, dns, k);
                const int ob = 2 * (__mul24(__mul24(jj - k, R) + k, S) + t) + part;
                // the table holds -sin: B = -(sine product)
                const float sg = part ? 1.f : -1.f;
#pragma unroll
                for (int v = 0; v < 4; ++v) {
                    const int q = (qb << 4) + 4 * kk + v;
                    if (q <= h) {
                        const float a = y0[i] + dc[i][v], b = sg * ds[i][v];
                        fb[ob + 2 * __mul24(q, NsS)] = a + b;
                        if (q) fb[ob + 2 * __mul24(R - q, NsS)] = a - b;
                    }
                }
            }
        }
    }
    __syncthreads();
}

// Forward DFTs of nb = 2^lgnb sequences of length d->n, element i of
// sequence t at buf[i S + t]. The stage twiddles and prime-radix matrices are
// read from the pool (each butterfly reads R - 1 consecutive twiddles, shared
// by every workgroup of the same length, so they stay in the caches). The
// plan guarantees that every prime-radix stage's result tiles fit the
// workgroup. Ends with a barrier when there is a stage.
// `stw` points at this length's stage twiddles: pool + d->stw, or a copy
// of them (d->ntw values) in LDS.
template <int NT, int EPT>
__device__ __forceinline__ void lds_fft(float2* buf, int S, int lgnb, const FftDesc* __restrict__ d,
                                        const float2* __restrict__ pool, const float2* __restrict__ stw) {
    const int n = d->n;
    const int ns = d->nstages;
    int Ns = 1;
    for (int s = 0; s < ns; ++s) {
        const int R = d->radix[s];
        const float rns = d->rcp_ns[s];
        const float2* tw = stw + d->stoff[s];
        switch (R) {
            case 2: stage_fixed<2, NT, EPT>(buf, n, S, lgnb, Ns, rns, tw); break;
            case 3: stage_fixed<3, NT, EPT>(buf, n, S, lgnb, Ns, rns, tw); break;
            case 4: stage_fixed<4, NT, EPT>(buf, n, S, lgnb, Ns, rns, tw); break;
            case 5: stage_fixed<5, NT, EPT>(buf, n, S, lgnb, Ns, rns, tw); break;
            case 6: stage_fixed<6, NT, EPT>(buf, n, S, lgnb, Ns, rns, tw); break;
            case 7: stage_fixed<7, NT, EPT>(buf, n, S, lgnb, Ns, rns, tw); break;
            case 8: stage_fixed<8, NT, EPT>(buf, n, S, lgnb, Ns, rns, tw); break;
            case 9: stage_fixed<9, NT, EPT>(buf, n, S, lgnb, Ns, rns, tw); break;
            case 10: stage_fixed<10, NT, EPT>(buf, n, S, lgnb, Ns, rns, tw); break;
            case 11: stage_fixed<11, NT, EPT>(buf, n, S, lgnb, Ns, rns, tw); break;
            case 12: stage_fixed<12, NT, EPT>(buf, n, S, lgnb, Ns, rns, tw); break;
            case 13: stage_fixed<13, NT, EPT>(buf, n, S, lgnb, Ns, rns, tw); break;
            case 14: stage_fixed<14, NT, EPT>(buf, n, S, lgnb, Ns, rns, tw); break;
            case 15: stage_fixed<15, NT, EPT>(buf, n, S, lgnb, Ns, rns, tw); break;
            case 16: stage_fixed<16, NT, EPT>(buf, n, S, lgnb, Ns, rns, tw); break;
            default:
                stage_prime_mfma<NT>(buf, n, S, lgnb, Ns, R, rns, d->rcp_h[s], tw, pool + d->full);
                break;
        }
        Ns *= R;
    }
}

template <int NT, int EPT>
__device__ __forceinline__ void lds_fft(float2* buf, int S, int lgnb, const FftDesc* __restrict__ d,
                                        const float2* __restrict__ pool) {
    lds_fft<NT, EPT>(buf, S, lgnb, d, pool, pool + d->stw);
}

// Interleave stride of nb = 2^lgnb sequences.
__host__ __device__ __forceinline__ int seq_stride(int lgnb) { return lgnb ? (1 << lgnb) + 1 : 1; }

}  // namespace nsg
