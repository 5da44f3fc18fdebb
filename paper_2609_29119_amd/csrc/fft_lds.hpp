// In-LDS mixed-radix Stockham FFT for one workgroup (gfx950, wave64).
//
// A workgroup of NT threads transforms `nb` independent sequences of length n
// stored at buf + t*ld (t < nb) in place. Each stage with radix R reads every
// butterfly's R inputs into registers, synchronises, then applies the stage
// twiddles, the length-R DFT and writes the outputs in autosort order, so one
// LDS buffer suffices. The caller guarantees nb*n <= NT*EPT, which bounds the
// registers every thread needs per stage.
//
// All transforms are forward DFTs (eq. 1, exp(-2 pi i k j / n)); inverse
// transforms are obtained by conjugating input and output.
#pragma once

#include <hip/hip_runtime.h>

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

// ---------------------------------------------------------------- butterflies
// Forward DFTs of length R on v[0..R-1], in place.

template <int R> struct Dft;

template <> struct Dft<2> {
    __device__ __forceinline__ static void run(float2* v) {
        const float2 a = v[0], b = v[1];
        v[0] = cadd(a, b);
        v[1] = csub(a, b);
    }
};

template <> struct Dft<3> {
    __device__ __forceinline__ static void run(float2* v) {
        constexpr float s = 0.8660254037844386467637f;   // sin(2 pi / 3)
        const float2 t1 = cadd(v[1], v[2]);
        const float2 t2 = make_float2(v[0].x - 0.5f * t1.x, v[0].y - 0.5f * t1.y);
        const float2 d = csub(v[1], v[2]);
        const float2 t3 = make_float2(s * d.y, -s * d.x);   // -i s (v1 - v2)
        v[0] = cadd(v[0], t1);
        v[1] = cadd(t2, t3);
        v[2] = csub(t2, t3);
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

// Odd R: pair outputs q and R-q. With s_r = v_r + v_{R-r}, d_r = v_r - v_{R-r}:
//   X_q     = v_0 + sum_r s_r cos(2 pi r q/R) - i sum_r d_r sin(2 pi r q/R)
//   X_{R-q} = v_0 + sum_r s_r cos(2 pi r q/R) + i sum_r d_r sin(2 pi r q/R)
template <int R> struct OddConst;
template <> struct OddConst<5> {
    __device__ __forceinline__ static float c(int t) {
        return t == 1 ? 0.3090169943749474241023f : -0.8090169943749474241023f;
    }
    __device__ __forceinline__ static float s(int t) {
        return t == 1 ? 0.9510565162951535721164f : 0.5877852522924731291687f;
    }
};
template <> struct OddConst<7> {
    __device__ __forceinline__ static float c(int t) {
        return t == 1 ? 0.623489801858733530525f : (t == 2 ? -0.2225209339563144042889f : -0.9009688679024191262361f);
    }
    __device__ __forceinline__ static float s(int t) {
        return t == 1 ? 0.7818314824680298087084f : (t == 2 ? 0.9749279121818236070181f : 0.4338837391175581204758f);
    }
};

template <int R> struct DftOdd {
    __device__ __forceinline__ static void run(float2* v) {
        constexpr int h = (R - 1) / 2;
        float2 s[h + 1], d[h + 1];
#pragma unroll
        for (int r = 1; r <= h; ++r) {
            s[r] = cadd(v[r], v[R - r]);
            d[r] = csub(v[r], v[R - r]);
        }
        float2 x0 = v[0];
#pragma unroll
        for (int r = 1; r <= h; ++r) x0 = cadd(x0, s[r]);
#pragma unroll
        for (int q = 1; q <= h; ++q) {
            float2 A = v[0], B = make_float2(0.f, 0.f);
#pragma unroll
            for (int r = 1; r <= h; ++r) {
                const int t = (r * q) % R;
                // cos(2 pi t / R) = c(min(t, R-t)); sin = +s for t <= h, -s otherwise
                const int u = t <= h ? t : R - t;
                const float cs = OddConst<R>::c(u);
                const float sn = t <= h ? OddConst<R>::s(u) : -OddConst<R>::s(u);
                A.x += s[r].x * cs; A.y += s[r].y * cs;
                B.x += d[r].x * sn; B.y += d[r].y * sn;
            }
            v[q] = make_float2(A.x + B.y, A.y - B.x);       // A - i B
            v[R - q] = make_float2(A.x - B.y, A.y + B.x);   // A + i B
        }
        v[0] = x0;
    }
};
template <> struct Dft<5> { __device__ __forceinline__ static void run(float2* v) { DftOdd<5>::run(v); } };
template <> struct Dft<7> { __device__ __forceinline__ static void run(float2* v) { DftOdd<7>::run(v); } };

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

// LDS slot of element i: one pad slot after every 8 complex values, which
// breaks the power-of-two strides of Stockham writes across the banks.
__device__ __forceinline__ int lp(int i) { return i + (i >> 3); }

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

// Stage twiddle omega_n^t from the two-level table in LDS: hi values at
// twl[0 .. nhi), lo values at twl[nhi .. nhi + 2^lg).
struct TwL {
    const float2* t;
    int nhi;
    int lg;
};
__device__ __forceinline__ float2 tw_at(const TwL& w, int t) {
    return cmul(w.t[t >> w.lg], w.t[w.nhi + (t & ((1 << w.lg) - 1))]);
}

// Odd prime radix with the symmetric pairing of DftOdd; cos/sin of 2 pi u/R
// are read from the twiddle table (tw[u m] = omega_R^u), a uniform address.
template <int R> struct DftOddT {
    __device__ __forceinline__ static void run(float2* v, const float2* __restrict__ tw, int m) {
        constexpr int h = (R - 1) / 2;
        float cs[h + 1], sn[h + 1];
#pragma unroll
        for (int u = 1; u <= h; ++u) {
            const float2 w = tw[u * m];
            cs[u] = w.x;
            sn[u] = -w.y;
        }
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
                const int t = (r * q) % R;
                const int u = t <= h ? t : R - t;
                const float c = cs[u];
                const float sg = t <= h ? sn[u] : -sn[u];
                A.x += s[r].x * c; A.y += s[r].y * c;
                B.x += d[r].x * sg; B.y += d[r].y * sg;
            }
            v[q] = make_float2(A.x + B.y, A.y - B.x);
            v[R - q] = make_float2(A.x - B.y, A.y + B.x);
        }
        v[0] = x0;
    }
};

template <int R> struct Radix {
    __device__ __forceinline__ static void run(float2* v, const float2* __restrict__, int) { Dft<R>::run(v); }
};
template <> struct Radix<11> { __device__ __forceinline__ static void run(float2* v, const float2* tw, int m) { DftOddT<11>::run(v, tw, m); } };
template <> struct Radix<13> { __device__ __forceinline__ static void run(float2* v, const float2* tw, int m) { DftOddT<13>::run(v, tw, m); } };

// -------------------------------------------------------------------- stages

// Stockham stage with compile-time radix R over nb sequences of length n at
// LDS slots lp(t*ld + i). Butterfly jj of sequence t reads in[jj + r m]
// (m = n/R), multiplies input r by omega_{Ns R}^{r k} (k = jj mod Ns), applies
// the length-R DFT, and after a barrier writes out[(jj - k) R + k + r Ns].
template <int R, int NT, int EPT>
__device__ __forceinline__ void stage_fixed(float2* buf, int nb, int ld, int n, int Ns,
                                            const float2* __restrict__ tw, const TwL& twl) {
    constexpr int BPT = (EPT + R - 1) / R;
    const int tid = stage_tid();
    const int m = n / R;
    const int total = __mul24(nb, m);
    const int stride = n / (Ns * R);
    const Div dm = mkdiv(m), dns = mkdiv(Ns);
    float2 v[BPT][R];
    int ob[BPT];
#pragma unroll
    for (int b = 0; b < BPT; ++b) {
        const int j = tid + b * NT;
        ob[b] = -1;
        if (j < total) {
            int jj = j, t = 0, k = 0;
            if (nb > 1) t = qdiv(j, dm, jj);
            if (Ns > 1) qdiv(jj, dns, k);
            const int base = __mul24(t, ld);
            int a = base + jj;
#pragma unroll
            for (int r = 0; r < R; ++r) {
                v[b][r] = buf[lp(a)];
                a += m;
            }
            if (Ns > 1) {
                const int step = __mul24(k, stride);
                int ti = step;
#pragma unroll
                for (int r = 1; r < R; ++r) {
                    v[b][r] = cmul(v[b][r], tw_at(twl, ti));
                    ti += step;
                }
            }
            Radix<R>::run(v[b], tw, m);
            ob[b] = base + (jj - k) * R + k;
        }
    }
    __syncthreads();
#pragma unroll
    for (int b = 0; b < BPT; ++b) {
        if (ob[b] >= 0) {
            int a = ob[b];
#pragma unroll
            for (int r = 0; r < R; ++r) {
                buf[lp(a)] = v[b][r];
                a += Ns;
            }
        }
    }
    __syncthreads();
}

// Stockham stage for an odd prime radix R (17 <= R <= kGenericMaxRadix) known
// only at run time. Inputs are first multiplied by their stage twiddles in
// place; then each work item (butterfly, q) produces the output pair q, R-q by
// the symmetric sums of DftOdd, reading the twiddled inputs from LDS.
template <int NT, int EPT>
__device__ __forceinline__ void stage_generic(float2* buf, int nb, int ld, int n, int Ns, int R,
                                              const float2* __restrict__ tw, const TwL& twl, float2* wr) {
    constexpr int IPT = (EPT * 6 + 9) / 10;   // items <= nb n (R+1)/(2R) <= 0.55 NT EPT
    const int tid = stage_tid();
    const int m = n / R;
    const int h = (R - 1) >> 1;
    const int stride = n / (Ns * R);
    const Div dn = mkdiv(n), dm = mkdiv(m), dns = mkdiv(Ns), dhp = mkdiv(h + 1);
    for (int t = tid; t < R; t += NT) wr[t] = tw[t * m];   // omega_R^t
    if (Ns > 1) {
        const int tot = __mul24(nb, n);
        for (int e = tid; e < tot; e += NT) {
            int i = e, jj, k, t = 0;
            if (nb > 1) t = qdiv(e, dn, i);
            const int r = qdiv(i, dm, jj);
            if (r) {
                qdiv(jj, dns, k);
                const int a = lp(__mul24(t, ld) + i);
                buf[a] = cmul(buf[a], tw_at(twl, __mul24(__mul24(r, k), stride)));
            }
        }
    }
    __syncthreads();
    const int hp = h + 1;
    const int items = nb * m * hp;
    float2 o0[IPT], o1[IPT];
    int ob[IPT], oq[IPT];
#pragma unroll
    for (int b = 0; b < IPT; ++b) {
        const int it = tid + b * NT;
        ob[b] = -1;
        if (it < items) {
            int q, jj, k = 0, t = 0;
            const int j = qdiv(it, dhp, q);
            jj = j;
            if (nb > 1) t = qdiv(j, dm, jj);
            if (Ns > 1) qdiv(jj, dns, k);
            const int src = __mul24(t, ld) + jj;
            float2 A = buf[lp(src)], B = make_float2(0.f, 0.f);
            int idx = 0;
            int ia = src, ic = src + __mul24(R, m);
            for (int r = 1; r <= h; ++r) {
                idx += q;
                if (idx >= R) idx -= R;
                ia += m;
                ic -= m;
                const float2 a = buf[lp(ia)], c = buf[lp(ic)];
                const float2 w = wr[idx];        // (cos, -sin) of 2 pi idx / R
                A.x += (a.x + c.x) * w.x;
                A.y += (a.y + c.y) * w.x;
                B.x -= (a.x - c.x) * w.y;
                B.y -= (a.y - c.y) * w.y;
            }
            o0[b] = make_float2(A.x + B.y, A.y - B.x);
            o1[b] = make_float2(A.x - B.y, A.y + B.x);
            ob[b] = __mul24(t, ld) + __mul24(jj - k, R) + k;
            oq[b] = q;
        }
    }
    __syncthreads();
#pragma unroll
    for (int b = 0; b < IPT; ++b) {
        if (ob[b] >= 0) {
            buf[lp(ob[b] + __mul24(oq[b], Ns))] = o0[b];
            if (oq[b]) buf[lp(ob[b] + __mul24(R - oq[b], Ns))] = o1[b];
        }
    }
    __syncthreads();
}

// Forward DFTs of nb sequences of length d->n at LDS slots lp(t*ld + i). `wr`
// is LDS scratch for kGenericMaxRadix complex values and `twlds` for kTwSlots.
// Ends with a barrier (when there is at least one stage).
template <int NT, int EPT>
__device__ __forceinline__ void lds_fft(float2* buf, int nb, int ld, const FftDesc* __restrict__ d,
                                        const float2* __restrict__ twpool, float2* wr, float2* twlds) {
    const int n = d->n;
    const int ns = d->nstages;
    const float2* tw = twpool + d->tw;
    // the first stage (Ns = 1) needs no twiddles and ends with a barrier, so
    // the table is visible from the second stage on
    const TwL twl{twlds, d->nhi, d->lg};
    for (int i = threadIdx.x; i < d->nhi + (1 << d->lg); i += NT) twlds[i] = tw[n + i];
    int Ns = 1;
    for (int s = 0; s < ns; ++s) {
        const int R = d->radix[s];
        switch (R) {
            case 8: stage_fixed<8, NT, EPT>(buf, nb, ld, n, Ns, tw, twl); break;
            case 4: stage_fixed<4, NT, EPT>(buf, nb, ld, n, Ns, tw, twl); break;
            case 2: stage_fixed<2, NT, EPT>(buf, nb, ld, n, Ns, tw, twl); break;
            case 3: stage_fixed<3, NT, EPT>(buf, nb, ld, n, Ns, tw, twl); break;
            case 5: stage_fixed<5, NT, EPT>(buf, nb, ld, n, Ns, tw, twl); break;
            case 7: stage_fixed<7, NT, EPT>(buf, nb, ld, n, Ns, tw, twl); break;
            case 11: stage_fixed<11, NT, EPT>(buf, nb, ld, n, Ns, tw, twl); break;
            case 13: stage_fixed<13, NT, EPT>(buf, nb, ld, n, Ns, tw, twl); break;
            default: stage_generic<NT, EPT>(buf, nb, ld, n, Ns, R, tw, twl, wr); break;
        }
        Ns *= R;
    }
}

}  // namespace nsg
