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

// -------------------------------------------------------------------- stages

// Stockham stage with compile-time radix R. Butterfly jj of transform t reads
// in[jj + r m] (m = n/R), multiplies input r by omega_{Ns R}^{r k} (k = jj mod Ns),
// and writes out[(jj - k) R + k + r Ns].
template <int R, int NT, int EPT>
__device__ __forceinline__ void stage_fixed(float2* buf, int nb, int ld, int n, int Ns,
                                            const float2* __restrict__ tw) {
    constexpr int BPT = (EPT + R - 1) / R;
    const int m = n / R;
    const int total = nb * m;
    const int stride = n / (Ns * R);
    float2 v[BPT][R];
#pragma unroll
    for (int b = 0; b < BPT; ++b) {
        const int j = threadIdx.x + b * NT;
        if (j < total) {
            const int t = j / m;
            const int jj = j - t * m;
            const float2* src = buf + t * ld + jj;
#pragma unroll
            for (int r = 0; r < R; ++r) v[b][r] = src[r * m];
        }
    }
    __syncthreads();
#pragma unroll
    for (int b = 0; b < BPT; ++b) {
        const int j = threadIdx.x + b * NT;
        if (j < total) {
            const int t = j / m;
            const int jj = j - t * m;
            const int k = jj % Ns;
            if (Ns > 1) {
#pragma unroll
                for (int r = 1; r < R; ++r) v[b][r] = cmul(v[b][r], tw[r * k * stride]);
            }
            Dft<R>::run(v[b]);
            float2* dst = buf + t * ld + (jj - k) * R + k;
#pragma unroll
            for (int r = 0; r < R; ++r) dst[r * Ns] = v[b][r];
        }
    }
    __syncthreads();
}

// Stockham stage for an odd prime radix R (11 <= R <= kGenericMaxRadix) known
// only at run time. Inputs are first multiplied by their stage twiddles in
// place; then each work item (butterfly, q) produces the output pair q, R-q by
// the symmetric sums of DftOdd, reading the twiddled inputs from LDS.
template <int NT, int EPT>
__device__ __forceinline__ void stage_generic(float2* buf, int nb, int ld, int n, int Ns, int R,
                                           const float2* __restrict__ tw, float2* wr) {
    constexpr int IPT = (EPT * 6 + 9) / 10;   // items <= nb n (R+1)/(2R) <= 0.55 NT EPT
    const int m = n / R;
    const int h = (R - 1) >> 1;
    const int stride = n / (Ns * R);
    for (int t = threadIdx.x; t < R; t += NT) wr[t] = tw[t * m];   // omega_R^t
    if (Ns > 1) {
        const int tot = nb * n;
        for (int e = threadIdx.x; e < tot; e += NT) {
            const int t = e / n;
            const int i = e - t * n;
            const int r = i / m;
            if (r) {
                const int k = (i - r * m) % Ns;
                float2* p = buf + t * ld + i;
                *p = cmul(*p, tw[r * k * stride]);
            }
        }
    }
    __syncthreads();
    const int hp = h + 1;
    const int items = nb * m * hp;
    float2 o0[IPT], o1[IPT];
#pragma unroll
    for (int b = 0; b < IPT; ++b) {
        const int it = threadIdx.x + b * NT;
        if (it < items) {
            const int q = it % hp;
            const int j = it / hp;
            const int t = j / m;
            const int jj = j - t * m;
            const float2* src = buf + t * ld + jj;
            float2 A = src[0], B = make_float2(0.f, 0.f);
            int idx = 0;
            for (int r = 1; r <= h; ++r) {
                idx += q;
                if (idx >= R) idx -= R;
                const float2 a = src[r * m], c = src[(R - r) * m];
                const float2 w = wr[idx];        // (cos, -sin) of 2 pi idx / R
                A.x += (a.x + c.x) * w.x;
                A.y += (a.y + c.y) * w.x;
                B.x -= (a.x - c.x) * w.y;
                B.y -= (a.y - c.y) * w.y;
            }
            o0[b] = make_float2(A.x + B.y, A.y - B.x);
            o1[b] = make_float2(A.x - B.y, A.y + B.x);
        }
    }
    __syncthreads();
#pragma unroll
    for (int b = 0; b < IPT; ++b) {
        const int it = threadIdx.x + b * NT;
        if (it < items) {
            const int q = it % hp;
            const int j = it / hp;
            const int t = j / m;
            const int jj = j - t * m;
            const int k = jj % Ns;
            float2* dst = buf + t * ld + (jj - k) * R + k;
            dst[q * Ns] = o0[b];
            if (q) dst[(R - q) * Ns] = o1[b];
        }
    }
    __syncthreads();
}

// Forward DFTs of nb sequences of length d->n at buf + t*ld. `wr` is LDS
// scratch for kGenericMaxRadix complex values. Ends with a barrier (when
// there is at least one stage).
template <int NT, int EPT>
__device__ __forceinline__ void lds_fft(float2* buf, int nb, int ld, const FftDesc* __restrict__ d,
                        const float2* __restrict__ twpool, float2* wr) {
    const int n = d->n;
    const int ns = d->nstages;
    const float2* tw = twpool + d->tw;
    int Ns = 1;
    for (int s = 0; s < ns; ++s) {
        const int R = d->radix[s];
        switch (R) {
            case 8: stage_fixed<8, NT, EPT>(buf, nb, ld, n, Ns, tw); break;
            case 4: stage_fixed<4, NT, EPT>(buf, nb, ld, n, Ns, tw); break;
            case 2: stage_fixed<2, NT, EPT>(buf, nb, ld, n, Ns, tw); break;
            case 3: stage_fixed<3, NT, EPT>(buf, nb, ld, n, Ns, tw); break;
            case 5: stage_fixed<5, NT, EPT>(buf, nb, ld, n, Ns, tw); break;
            case 7: stage_fixed<7, NT, EPT>(buf, nb, ld, n, Ns, tw); break;
            default: stage_generic<NT, EPT>(buf, nb, ld, n, Ns, R, tw, wr); break;
        }
        Ns *= R;
    }
}

}  // namespace nsg
