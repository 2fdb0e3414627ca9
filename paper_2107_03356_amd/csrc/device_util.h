// Device helpers shared by the streaming kernels (pass.hip, static_query.hip).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mfac {
namespace {

typedef float f4v __attribute__((ext_vector_type(4)));

// Window rows are read exactly once per pass: nontemporal loads stream them
// past the caches (measured +15-20% HBM throughput on gfx950 for these passes).
__device__ __forceinline__ float4 ld_stream(const float* __restrict__ p) {
    const f4v v = __builtin_nontemporal_load(reinterpret_cast<const f4v*>(p));
    return make_float4(v.x, v.y, v.z, v.w);
}

__device__ __forceinline__ float4 ld4(const float* __restrict__ p, int64_t j, int64_t d, int aligned) {
    if (aligned && j + 3 < d) return *reinterpret_cast<const float4*>(p + j);
    float4 r;
    r.x = (j < d) ? p[j] : 0.f;
    r.y = (j + 1 < d) ? p[j + 1] : 0.f;
    r.z = (j + 2 < d) ? p[j + 2] : 0.f;
    r.w = (j + 3 < d) ? p[j + 3] : 0.f;
    return r;
}

__device__ __forceinline__ void st4(float* __restrict__ p, int64_t j, int64_t d, int aligned, float4 v) {
    if (aligned && j + 3 < d) {
        *reinterpret_cast<float4*>(p + j) = v;
        return;
    }
    if (j < d) p[j] = v.x;
    if (j + 1 < d) p[j + 1] = v.y;
    if (j + 2 < d) p[j + 2] = v.z;
    if (j + 3 < d) p[j + 3] = v.w;
}

// Pass outputs are written once and not read back by the pass: nontemporal
// stores keep them from competing with the window stream for the caches
// (the one-vector pass 2 over a 105 GB window: 15.2 -> 14.8 ms on gfx950).
__device__ __forceinline__ void st_stream(float* __restrict__ p, float4 v) {
    const f4v w = {v.x, v.y, v.z, v.w};
    __builtin_nontemporal_store(w, reinterpret_cast<f4v*>(p));
}

// st4 with a nontemporal store for the aligned, in-range case.
__device__ __forceinline__ void st4_stream(float* __restrict__ p, int64_t j, int64_t d, int aligned, float4 v) {
    if (aligned && j + 3 < d) {
        st_stream(p + j, v);
        return;
    }
    st4(p, j, d, aligned, v);
}

__device__ __forceinline__ float dot4(float4 a, float4 b, float s) {
    s = fmaf(a.x, b.x, s);
    s = fmaf(a.y, b.y, s);
    s = fmaf(a.z, b.z, s);
    s = fmaf(a.w, b.w, s);
    return s;
}

// fp64 dot of two fp32 float4 (the products are exact in fp64)
__device__ __forceinline__ double dot4d(float4 a, float4 b, double s) {
    s = fma((double)a.x, (double)b.x, s);
    s = fma((double)a.y, (double)b.y, s);
    s = fma((double)a.z, (double)b.z, s);
    s = fma((double)a.w, (double)b.w, s);
    return s;
}

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, 64);
    return x;
}

// Sum N per-lane values over the 64 lanes of a wave in about N + 5 shuffles
// (instead of 6 N): at each halving step a lane keeps half of its pending sums
// and trades the other half with its partner lane (lane ^ O), so the number of
// pending values halves while the lanes covered double. Once one value is
// left, plain butterfly steps finish the sum. On return the lane holds the
// total of value `base`; exactly one lane per value has writer == true.
template <typename T, int N, int C, int O>
struct WaveReduceMany {
    static __device__ __forceinline__ void run(T (&s)[N], int lane, int& base, int& creal, bool& dup) {
        if constexpr (O > 0) {
            const bool up = (lane & O) != 0;
            if constexpr (C > 1) {
                constexpr int H = (C + 1) / 2;
#pragma unroll
                for (int j = 0; j < H; ++j) {
                    const T lo = s[j];
                    const T hi = (H + j < C) ? s[(H + j < N) ? H + j : N - 1] : T(0);
                    const T send = up ? lo : hi;
                    const T keep = up ? hi : lo;
                    s[j] = keep + __shfl_xor(send, O, 64);
                }
                base += up ? H : 0;
                creal = up ? (creal > H ? creal - H : 0) : (creal < H ? creal : H);
                WaveReduceMany<T, N, H, O / 2>::run(s, lane, base, creal, dup);
            } else {
                s[0] += __shfl_xor(s[0], O, 64);
                dup = dup || up;
                WaveReduceMany<T, N, 1, O / 2>::run(s, lane, base, creal, dup);
            }
        }
    }
};

template <int N, typename T>
__device__ __forceinline__ T wave_reduce_many(T (&s)[N], int lane, int& base, bool& writer) {
    base = 0;
    int creal = N;
    bool dup = false;
    WaveReduceMany<T, N, N, 32>::run(s, lane, base, creal, dup);
    writer = !dup && creal > 0;
    return s[0];
}

}  // namespace
}  // namespace mfac
