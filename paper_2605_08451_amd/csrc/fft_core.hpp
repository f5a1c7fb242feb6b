// fft_core.hpp -- register-resident small DFTs for gfx950 (fp32 complex).
//
// dft<R, S>(v) replaces v[0..R) by its R-point DFT with kernel
// exp(S * 2 pi i n k / R) (S = -1 forward, +1 inverse, unnormalised), natural
// order in and out.  Sizes 2, 3, 4, 5 are written out; 6, 8, 9, 10, 12, 15, 16 are split
// R = A * B by decimation in time with compile-time twiddles, so after
// unrolling every index is a constant and the values stay in VGPRs.
#pragma once

#include <hip/hip_runtime.h>

namespace rubiconv {

__device__ __forceinline__ float2 cadd(float2 a, float2 b) { return make_float2(a.x + b.x, a.y + b.y); }
__device__ __forceinline__ float2 csub(float2 a, float2 b) { return make_float2(a.x - b.x, a.y - b.y); }
__device__ __forceinline__ float2 cmul(float2 a, float2 b) {
    return make_float2(a.x * b.x - a.y * b.y, a.x * b.y + a.y * b.x);
}
__device__ __forceinline__ float2 cconj(float2 a) { return make_float2(a.x, -a.y); }
__device__ __forceinline__ float2 cscale(float2 a, float s) { return make_float2(a.x * s, a.y * s); }
// multiply by S*i
template <int S>
__device__ __forceinline__ float2 mul_si(float2 a) {
    return S < 0 ? make_float2(a.y, -a.x) : make_float2(-a.y, a.x);
}

// ---------------------------------------------------------------- constants
// cos/sin of 2*pi*e/n evaluated in double at compile time (Taylor series after
// reduction to [-pi, pi]); exact enough that the float rounding dominates.
constexpr double kPi = 3.14159265358979323846264338327950288;
constexpr double taylor_sin(double x) {
    double term = x, sum = x;
    for (int k = 1; k < 30; ++k) {
        term *= -x * x / ((2.0 * k) * (2.0 * k + 1.0));
        sum += term;
    }
    return sum;
}
constexpr double taylor_cos(double x) {
    double term = 1.0, sum = 1.0;
    for (int k = 1; k < 30; ++k) {
        term *= -x * x / ((2.0 * k - 1.0) * (2.0 * k));
        sum += term;
    }
    return sum;
}
constexpr double reduced_angle(int e, int n) {
    // 2*pi*e/n reduced to (-pi, pi]
    int r = e % n;
    if (2 * r > n) r -= n;
    return 2.0 * kPi * static_cast<double>(r) / static_cast<double>(n);
}

template <int N>
struct RootTable {
    float c[N];
    float s[N];
    constexpr RootTable() : c(), s() {
        for (int e = 0; e < N; ++e) {
            c[e] = static_cast<float>(taylor_cos(reduced_angle(e, N)));
            s[e] = static_cast<float>(taylor_sin(reduced_angle(e, N)));
        }
    }
};

// v * exp(S * 2 pi i e / N) with e a compile-time constant after unrolling
template <int N, int S>
__device__ __forceinline__ float2 twiddle_const(float2 v, int e) {
    constexpr RootTable<N> t{};
    e %= N;
    if (e == 0) return v;
    if (2 * e == N) return make_float2(-v.x, -v.y);
    if (4 * e == N) return mul_si<S>(v);
    if (4 * e == 3 * N) return mul_si<-S>(v);
    const float2 w = make_float2(t.c[e], S * t.s[e]);
    return cmul(v, w);
}

// ---------------------------------------------------------------- small DFTs
template <int R, int S>
struct Dft;

template <int S>
struct Dft<1, S> {
    __device__ __forceinline__ static void run(float2 (&)[1]) {}
};

template <int S>
struct Dft<2, S> {
    __device__ __forceinline__ static void run(float2 (&v)[2]) {
        float2 a = v[0], b = v[1];
        v[0] = cadd(a, b);
        v[1] = csub(a, b);
    }
};

template <int S>
struct Dft<3, S> {
    __device__ __forceinline__ static void run(float2 (&v)[3]) {
        constexpr float kHalfSqrt3 = 0.866025403784438646763723170752936183f;
        float2 t1 = cadd(v[1], v[2]);
        float2 t2 = csub(v[1], v[2]);
        float2 m = make_float2(v[0].x - 0.5f * t1.x, v[0].y - 0.5f * t1.y);
        float2 r = mul_si<S>(cscale(t2, kHalfSqrt3));
        v[0] = cadd(v[0], t1);
        v[1] = cadd(m, r);
        v[2] = csub(m, r);
    }
};

template <int S>
struct Dft<4, S> {
    __device__ __forceinline__ static void run(float2 (&v)[4]) {
        float2 s02 = cadd(v[0], v[2]), d02 = csub(v[0], v[2]);
        float2 s13 = cadd(v[1], v[3]), d13 = mul_si<S>(csub(v[1], v[3]));
        v[0] = cadd(s02, s13);
        v[2] = csub(s02, s13);
        v[1] = cadd(d02, d13);
        v[3] = csub(d02, d13);
    }
};

template <int S>
struct Dft<5, S> {
    __device__ __forceinline__ static void run(float2 (&v)[5]) {
        constexpr float c1 = 0.309016994374947424102293417182819059f;   // cos(2pi/5)
        constexpr float c2 = -0.809016994374947424102293417182819059f;  // cos(4pi/5)
        constexpr float s1 = 0.951056516295153572116439333379382143f;   // sin(2pi/5)
        constexpr float s2 = 0.587785252292473129168705954639072769f;   // sin(4pi/5)
        float2 t1 = cadd(v[1], v[4]), t2 = cadd(v[2], v[3]);
        float2 t3 = csub(v[1], v[4]), t4 = csub(v[2], v[3]);
        float2 a1 = make_float2(v[0].x + c1 * t1.x + c2 * t2.x, v[0].y + c1 * t1.y + c2 * t2.y);
        float2 a2 = make_float2(v[0].x + c2 * t1.x + c1 * t2.x, v[0].y + c2 * t1.y + c1 * t2.y);
        float2 b1 = mul_si<S>(make_float2(s1 * t3.x + s2 * t4.x, s1 * t3.y + s2 * t4.y));
        float2 b2 = mul_si<S>(make_float2(s2 * t3.x - s1 * t4.x, s2 * t3.y - s1 * t4.y));
        v[0] = cadd(v[0], cadd(t1, t2));
        v[1] = cadd(a1, b1);
        v[4] = csub(a1, b1);
        v[2] = cadd(a2, b2);
        v[3] = csub(a2, b2);
    }
};

// R = A * B, decimation in time: n = B*n1 + n2, k = k1 + A*k2,
// X[k1 + A k2] = sum_n2 w_B^(n2 k2) w_R^(n2 k1) sum_n1 w_A^(n1 k1) x[B n1 + n2].
template <int A, int B, int S>
struct DftSplit {
    __device__ __forceinline__ static void run(float2 (&v)[A * B]) {
        constexpr int R = A * B;
        float2 t[R];
#pragma unroll
        for (int n2 = 0; n2 < B; ++n2) {
            float2 s[A];
#pragma unroll
            for (int n1 = 0; n1 < A; ++n1) s[n1] = v[B * n1 + n2];
            Dft<A, S>::run(s);
#pragma unroll
            for (int k1 = 0; k1 < A; ++k1) t[k1 * B + n2] = twiddle_const<R, S>(s[k1], n2 * k1);
        }
#pragma unroll
        for (int k1 = 0; k1 < A; ++k1) {
            float2 s[B];
#pragma unroll
            for (int n2 = 0; n2 < B; ++n2) s[n2] = t[k1 * B + n2];
            Dft<B, S>::run(s);
#pragma unroll
            for (int k2 = 0; k2 < B; ++k2) v[k1 + A * k2] = s[k2];
        }
    }
};

template <int S>
struct Dft<6, S> {
    __device__ __forceinline__ static void run(float2 (&v)[6]) { DftSplit<2, 3, S>::run(v); }
};
template <int S>
struct Dft<9, S> {
    __device__ __forceinline__ static void run(float2 (&v)[9]) { DftSplit<3, 3, S>::run(v); }
};
template <int S>
struct Dft<10, S> {
    __device__ __forceinline__ static void run(float2 (&v)[10]) { DftSplit<2, 5, S>::run(v); }
};
template <int S>
struct Dft<12, S> {
    __device__ __forceinline__ static void run(float2 (&v)[12]) { DftSplit<4, 3, S>::run(v); }
};
template <int S>
struct Dft<15, S> {
    __device__ __forceinline__ static void run(float2 (&v)[15]) { DftSplit<3, 5, S>::run(v); }
};
template <int S>
struct Dft<8, S> {
    __device__ __forceinline__ static void run(float2 (&v)[8]) { DftSplit<2, 4, S>::run(v); }
};
template <int S>
struct Dft<16, S> {
    __device__ __forceinline__ static void run(float2 (&v)[16]) { DftSplit<4, 4, S>::run(v); }
};
template <int S>
struct Dft<20, S> {
    __device__ __forceinline__ static void run(float2 (&v)[20]) { DftSplit<4, 5, S>::run(v); }
};
template <int S>
struct Dft<24, S> {
    __device__ __forceinline__ static void run(float2 (&v)[24]) { DftSplit<8, 3, S>::run(v); }
};
template <int S>
struct Dft<25, S> {
    __device__ __forceinline__ static void run(float2 (&v)[25]) { DftSplit<5, 5, S>::run(v); }
};
template <int S>
struct Dft<30, S> {
    __device__ __forceinline__ static void run(float2 (&v)[30]) { DftSplit<6, 5, S>::run(v); }
};
template <int S>
struct Dft<32, S> {
    __device__ __forceinline__ static void run(float2 (&v)[32]) { DftSplit<8, 4, S>::run(v); }
};

// ---------------------------------------------------------------- spectral product
// Conjugate-symmetry separation (Appendix, dual real FFTs; Algorithm 3) fused with
// the product.  a is the pair transform at f = (u, v) with u <= N1/2, b at the
// frequency -f.  For the filter pair h_d + i h_{d+1}:
//     H_d = (a + conj b) / 2,   H_{d+1} = (a - conj b) / (2i),
// kept as S = c (H_d + H_{d+1}) and Df = c (H_d - H_{d+1}).  For the data pair the
// transform of y_d + i y_{d+1} is then
//     W(f)  = a S + conj(b) Df,   W(-f) = conj(conj(b) S + a Df).
__device__ __forceinline__ void filter_sdf(float2 a, float2 b, float c, float2& s, float2& df) {
    const float2 hd = make_float2(0.5f * (a.x + b.x), 0.5f * (a.y - b.y));
    const float2 hd1 = make_float2(0.5f * (a.y + b.y), 0.5f * (b.x - a.x));
    s = cscale(cadd(hd, hd1), c);
    df = cscale(csub(hd, hd1), c);
}
__device__ __forceinline__ float2 product_f(float2 a, float2 b, float2 s, float2 df) {
    return cadd(cmul(a, s), cmul(cconj(b), df));
}
__device__ __forceinline__ float2 product_neg_f(float2 a, float2 b, float2 s, float2 df) {
    return cconj(cadd(cmul(cconj(b), s), cmul(a, df)));
}

}  // namespace rubiconv
