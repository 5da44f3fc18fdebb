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

// Exact quotient and remainder of 0 <= x < 2^22 by 0 < d < 2^22 through a
// float reciprocal: the product is within one unit of x/d, fixed by one step.
struct Div {
    float r;
    int d;
};
__device__ __forceinline__ Div mkdiv(int d) { return Div{1.0f / static_cast<float>(d), d}; }
__device__ __forceinline__ int qdiv(int x, Div v, int& rem) {
    int q = static_cast<int>(static_cast<float>(x) * v.r);
    int r = x - __mul24(q, v.d);
    if (r < 0) { --q; r += v.d; }
    else if (r >= v.d) { ++q; r -= v.d; }
    rem = r;
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
__device__ __forceinline__ void stage_fixed(float2* buf, int n, int S, int lgnb, int Ns,
                                            const float2* __restrict__ tws) {
    constexpr int BPT = (EPT + R - 1) / R;
    const int tid = stage_tid();
    const int m = n / R;
    const int total = m << lgnb;
    const int nbm = (1 << lgnb) - 1;
    const int mS = __mul24(m, S), NsS = __mul24(Ns, S);
    const Div dns = mkdiv(Ns);
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

// Stockham stage for an odd prime radix R (17 <= R <= kGenericMaxRadix) known
// only at run time. First each pair of inputs (r, R-r) is twiddled and
// replaced in place by s_r = y_r + y_{R-r}, d_r = y_r - y_{R-r}; then each
// work item (butterfly, group of four q) forms the output pairs q, R-q of
// DftPrime from s, d and the table wr[t] = omega_R^t.
template <int NT, int EPT>
__device__ __forceinline__ void stage_generic(float2* buf, int n, int S, int lgnb, int Ns, int R,
                                              const float2* __restrict__ tws, float2* wr,
                                              const float2* __restrict__ full) {
    constexpr int IPT = (EPT + 4) / 5;   // items <= NT EPT (R + 7) / (8 R) <= 0.18 NT EPT
    const int tid = stage_tid();
    const int m = n / R;
    const int h = (R - 1) >> 1;
    const int nbm = (1 << lgnb) - 1;
    const int mS = __mul24(m, S), NsS = __mul24(Ns, S);
    const int totb = m << lgnb;
    const Div dns = mkdiv(Ns), dh = mkdiv(h);
    for (int t = tid; t < R; t += NT) wr[t] = full[__mul24(t, m)];
    for (int e = tid; e < __mul24(totb, h); e += NT) {
        int r1;
        const int j = qdiv(e, dh, r1);
        const int r = r1 + 1;
        const int t = j & nbm, jj = j >> lgnb;
        const int a0 = __mul24(jj, S) + t;
        const int ia = a0 + __mul24(r, mS), ic = a0 + __mul24(R - r, mS);
        float2 ya = buf[ia], yc = buf[ic];
        if (Ns > 1) {
            int k;
            qdiv(jj, dns, k);
            const float2* w = tws + __mul24(k, R - 1);
            ya = cmul(ya, w[r - 1]);
            yc = cmul(yc, w[R - r - 1]);
        }
        buf[ia] = cadd(ya, yc);
        buf[ic] = csub(ya, yc);
    }
    __syncthreads();
    const int ng = (h + 4) >> 2;   // groups of four q over 0..h
    const int items = __mul24(totb, ng);
    const Div dng = mkdiv(ng);
    float2 o[IPT][8];
    int ob[IPT], oq[IPT];
#pragma unroll
    for (int b = 0; b < IPT; ++b) {
        const int it = tid + b * NT;
        ob[b] = -1;
        if (it < items) {
            int g;
            const int j = qdiv(it, dng, g);
            const int t = j & nbm, jj = j >> lgnb;
            const int a0 = __mul24(jj, S) + t;
            const int q0 = g << 2;
            const float2 y0 = buf[a0];
            float2 A[4], B[4];
            int idx[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                A[u] = y0;
                B[u] = make_float2(0.f, 0.f);
                idx[u] = 0;
            }
            int ia = a0, ic = a0 + __mul24(R, mS);
            for (int r = 1; r <= h; ++r) {
                ia += mS;
                ic -= mS;
                const float2 sv = buf[ia], dv = buf[ic];
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    idx[u] += q0 + u;
                    if (idx[u] >= R) idx[u] -= R;
                    const float2 w = wr[idx[u]];          // (cos, -sin) of 2 pi idx / R
                    A[u].x += sv.x * w.x;
                    A[u].y += sv.y * w.x;
                    B[u].x -= dv.x * w.y;
                    B[u].y -= dv.y * w.y;
                }
            }
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                o[b][2 * u] = make_float2(A[u].x + B[u].y, A[u].y - B[u].x);       // X_q
                o[b][2 * u + 1] = make_float2(A[u].x - B[u].y, A[u].y + B[u].x);   // X_{R-q}
            }
            int k = 0;
            if (Ns > 1) qdiv(jj, dns, k);
            ob[b] = __mul24(__mul24(jj - k, R) + k, S) + t;
            oq[b] = q0;
        }
    }
    __syncthreads();
#pragma unroll
    for (int b = 0; b < IPT; ++b) {
        if (ob[b] >= 0) {
#pragma unroll
            for (int u = 0; u < 4; ++u) {
                const int q = oq[b] + u;
                if (q <= h) {
                    buf[ob[b] + __mul24(q, NsS)] = o[b][2 * u];
                    if (q) buf[ob[b] + __mul24(R - q, NsS)] = o[b][2 * u + 1];
                }
            }
        }
    }
    __syncthreads();
}

// Forward DFTs of nb = 2^lgnb sequences of length d->n, element i of
// sequence t at buf[i S + t]. `wr` is LDS scratch for kWrSlots values; the
// stage twiddles are read from the pool (each butterfly reads R - 1
// consecutive values, shared by every workgroup of the same length, so they
// stay in the caches). Ends with a barrier when there is a stage.
template <int NT, int EPT>
__device__ __forceinline__ void lds_fft(float2* buf, int S, int lgnb, const FftDesc* __restrict__ d,
                                        const float2* __restrict__ pool, float2* wr) {
    const int n = d->n;
    const int ns = d->nstages;
    const float2* full = pool + d->full;
    int Ns = 1;
    for (int s = 0; s < ns; ++s) {
        const int R = d->radix[s];
        const float2* tw = pool + d->stw + d->stoff[s];
        switch (R) {
            case 2: stage_fixed<2, NT, EPT>(buf, n, S, lgnb, Ns, tw); break;
            case 3: stage_fixed<3, NT, EPT>(buf, n, S, lgnb, Ns, tw); break;
            case 4: stage_fixed<4, NT, EPT>(buf, n, S, lgnb, Ns, tw); break;
            case 5: stage_fixed<5, NT, EPT>(buf, n, S, lgnb, Ns, tw); break;
            case 6: stage_fixed<6, NT, EPT>(buf, n, S, lgnb, Ns, tw); break;
            case 7: stage_fixed<7, NT, EPT>(buf, n, S, lgnb, Ns, tw); break;
            case 8: stage_fixed<8, NT, EPT>(buf, n, S, lgnb, Ns, tw); break;
            case 9: stage_fixed<9, NT, EPT>(buf, n, S, lgnb, Ns, tw); break;
            case 10: stage_fixed<10, NT, EPT>(buf, n, S, lgnb, Ns, tw); break;
            case 11: stage_fixed<11, NT, EPT>(buf, n, S, lgnb, Ns, tw); break;
            case 12: stage_fixed<12, NT, EPT>(buf, n, S, lgnb, Ns, tw); break;
            case 13: stage_fixed<13, NT, EPT>(buf, n, S, lgnb, Ns, tw); break;
            case 14: stage_fixed<14, NT, EPT>(buf, n, S, lgnb, Ns, tw); break;
            case 15: stage_fixed<15, NT, EPT>(buf, n, S, lgnb, Ns, tw); break;
            case 16: stage_fixed<16, NT, EPT>(buf, n, S, lgnb, Ns, tw); break;
            default: stage_generic<NT, EPT>(buf, n, S, lgnb, Ns, R, tw, wr, full); break;
        }
        Ns *= R;
    }
}

// Interleave stride of nb = 2^lgnb sequences.
__host__ __device__ __forceinline__ int seq_stride(int lgnb) { return lgnb ? (1 << lgnb) + 1 : 1; }

}  // namespace nsg
