// device.h -- small device helpers shared by the HIP kernels (wave64 reductions,
// numerically guarded log-sum-exp pieces, sequence-length clamping, XCD-aware block
// numbering).
#pragma once
#include <hip/hip_runtime.h>
#include <math.h>
#include <stdint.h>

namespace tsc {

constexpr int kWave = 64;

__device__ __forceinline__ int64_t clamp_len(const int32_t* lengths, int64_t b, int64_t N) {
    if (!lengths) return N;
    int64_t L = lengths[b];
    return L < 1 ? 1 : (L > N ? N : L);
}

__device__ __forceinline__ float wave_max(float x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x = fmaxf(x, __shfl_xor(x, o, kWave));
    return x;
}
__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, kWave);
    return x;
}
__device__ __forceinline__ double wave_max_d(double x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x = fmax(x, __shfl_xor(x, o, kWave));
    return x;
}
__device__ __forceinline__ double wave_sum_d(double x) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) x += __shfl_xor(x, o, kWave);
    return x;
}

// Hardware exp/log (v_exp_f32 / v_log_f32 are base 2).  Inputs of the callers are
// exponents <= 0 and sums >= 2^-80, so no denormal handling is needed.
__device__ __forceinline__ float fexp(float x) { return __builtin_amdgcn_exp2f(x * 1.4426950408889634f); }

// Raw buffer access to `n` floats at `base` (a workgroup-uniform pointer): loads take a
// per-lane 32-bit byte offset and a uniform byte offset held in a scalar register; an
// access past the n floats reads 0.  The descriptor's third word is the gfx9 raw-buffer
// format (no stride, no swizzle).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const float* base, int n) {
    return __builtin_amdgcn_make_buffer_rsrc((void*)base, (short)0, 4 * n, 0x00020000);
}
__device__ __forceinline__ float4 buffer_load4(__amdgpu_buffer_rsrc_t r, unsigned voff, int soff) {
    typedef int v4i __attribute__((ext_vector_type(4)));
    const v4i x = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
    return make_float4(__int_as_float(x.x), __int_as_float(x.y), __int_as_float(x.z), __int_as_float(x.w));
}
__device__ __forceinline__ void buffer_store4(float4 v, __amdgpu_buffer_rsrc_t r, unsigned voff, int soff) {
    typedef int v4i __attribute__((ext_vector_type(4)));
    const v4i x = {__float_as_int(v.x), __float_as_int(v.y), __float_as_int(v.z), __float_as_int(v.w)};
    __builtin_amdgcn_raw_buffer_store_b128(x, r, voff, soff, 0);
}
__device__ __forceinline__ float buffer_load1(__amdgpu_buffer_rsrc_t r, unsigned voff, int soff) {
    return __int_as_float(__builtin_amdgcn_raw_buffer_load_b32(r, voff, soff, 0));
}
__device__ __forceinline__ void buffer_store1(float v, __amdgpu_buffer_rsrc_t r, unsigned voff, int soff) {
    __builtin_amdgcn_raw_buffer_store_b32(__float_as_int(v), r, voff, soff, 0);
}
__device__ __forceinline__ float flog(float x) { return __builtin_amdgcn_logf(x) * 0.6931471805599453f; }

// Full-wave reductions with DPP inside each row of 16 lanes and readlane across the four
// rows: the result is wave-uniform and the order of operations is fixed (deterministic).
__device__ __forceinline__ float dpp_f(float x, int ctrl) {
    const int v = __float_as_int(x);
    switch (ctrl) {
        case 0xB1: return __int_as_float(__builtin_amdgcn_update_dpp(v, v, 0xB1, 0xF, 0xF, false));
        case 0x4E: return __int_as_float(__builtin_amdgcn_update_dpp(v, v, 0x4E, 0xF, 0xF, false));
        case 0x141: return __int_as_float(__builtin_amdgcn_update_dpp(v, v, 0x141, 0xF, 0xF, false));
        default: return __int_as_float(__builtin_amdgcn_update_dpp(v, v, 0x140, 0xF, 0xF, false));
    }
}
__device__ __forceinline__ float rl(float x, int lane) {
    return __int_as_float(__builtin_amdgcn_readlane(__float_as_int(x), lane));
}
__device__ __forceinline__ float wave_max_fast(float x) {
    x = fmaxf(x, dpp_f(x, 0xB1));   // lanes i ^ 1
    x = fmaxf(x, dpp_f(x, 0x4E));   // lanes i ^ 2
    x = fmaxf(x, dpp_f(x, 0x141));  // mirror within 8
    x = fmaxf(x, dpp_f(x, 0x140));  // mirror within 16
    return fmaxf(fmaxf(rl(x, 0), rl(x, 16)), fmaxf(rl(x, 32), rl(x, 48)));
}
// Maximum over the 32 lanes of the calling lane's half-wave (DPP inside each row of 16
// lanes, then one exchange between the two rows); every lane of the half gets it
__device__ __forceinline__ float half_max32(float x) {
    x = fmaxf(x, dpp_f(x, 0xB1));   // lanes i ^ 1
    x = fmaxf(x, dpp_f(x, 0x4E));   // lanes i ^ 2
    x = fmaxf(x, dpp_f(x, 0x141));  // mirror within 8
    x = fmaxf(x, dpp_f(x, 0x140));  // mirror within 16
    return fmaxf(x, __shfl_xor(x, 16, kWave));
}
__device__ __forceinline__ float wave_sum_fast(float x) {
    x += dpp_f(x, 0xB1);
    x += dpp_f(x, 0x4E);
    x += dpp_f(x, 0x141);
    x += dpp_f(x, 0x140);
    return (rl(x, 0) + rl(x, 16)) + (rl(x, 32) + rl(x, 48));
}

// Online log-sum-exp state: value = m + log(s).  m = -inf means the empty sum.
struct Lse {
    float m, s;
};
__device__ __forceinline__ Lse lse_empty() { return {-INFINITY, 0.f}; }
__device__ __forceinline__ Lse lse_push(Lse a, float x) {
    if (x == -INFINITY) return a;
    if (x <= a.m) {
        a.s += __expf(x - a.m);
    } else {
        a.s = (a.m == -INFINITY ? 0.f : a.s * __expf(a.m - x)) + 1.f;
        a.m = x;
    }
    return a;
}
__device__ __forceinline__ Lse lse_merge(Lse a, Lse b) {
    if (b.m == -INFINITY) return a;
    if (a.m == -INFINITY) return b;
    float m = fmaxf(a.m, b.m);
    return {m, a.s * __expf(a.m - m) + b.s * __expf(b.m - m)};
}
__device__ __forceinline__ float lse_value(Lse a) {
    return a.m == -INFINITY ? -INFINITY : a.m + __logf(a.s);
}
__device__ __forceinline__ Lse wave_lse(Lse a) {
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) {
        Lse b{__shfl_xor(a.m, o, kWave), __shfl_xor(a.s, o, kWave)};
        a = lse_merge(a, b);
    }
    return a;
}

// Block-wide max of a double over `nthreads` threads (blockDim.x, multiple of 64).
// `red` is __shared__ scratch of at least nthreads/64 doubles.  Ends with a barrier.
__device__ __forceinline__ double block_max_d(double x, double* red) {
    x = wave_max_d(x);
    const int w = threadIdx.x / kWave, nw = blockDim.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) red[w] = x;
    __syncthreads();
    double r = red[0];
    for (int i = 1; i < nw; ++i) r = fmax(r, red[i]);
    __syncthreads();
    return r;
}
__device__ __forceinline__ float block_max(float x, float* red) {
    x = wave_max(x);
    const int w = threadIdx.x / kWave, nw = blockDim.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) red[w] = x;
    __syncthreads();
    float r = red[0];
    for (int i = 1; i < nw; ++i) r = fmaxf(r, red[i]);
    __syncthreads();
    return r;
}
__device__ __forceinline__ Lse block_lse(Lse a, float* red) {
    a = wave_lse(a);
    const int w = threadIdx.x / kWave, nw = blockDim.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) { red[2 * w] = a.m; red[2 * w + 1] = a.s; }
    __syncthreads();
    Lse r{red[0], red[1]};
    for (int i = 1; i < nw; ++i) r = lse_merge(r, Lse{red[2 * i], red[2 * i + 1]});
    __syncthreads();
    return r;
}

// Shift used before exponentiating: the max, or 0 when everything is -inf (so that
// -inf - shift stays -inf instead of NaN).
__device__ __forceinline__ float safe_shift(float m) { return m == -INFINITY ? 0.f : m; }
__device__ __forceinline__ double safe_shift_d(double m) { return m == -INFINITY ? 0.0 : m; }

// Online log-sum-exp folded K values at a time: value = m + log(s), m = -inf while empty.
// One exp per value plus one per chunk (the rescale of the running sum).
// A double that every lane of the wave holds, moved to scalar registers (the first lane's)
__device__ __forceinline__ double uniform_d(double x) {
    const unsigned long long u = __double_as_longlong(x);
    const unsigned lo = __builtin_amdgcn_readfirstlane((unsigned)u);
    const unsigned hi = __builtin_amdgcn_readfirstlane((unsigned)(u >> 32));
    return __longlong_as_double(((unsigned long long)hi << 32) | lo);
}

template <int K>
__device__ __forceinline__ void lse_fold(float& m, float& s, const float (&x)[K]) {
    float cm = x[0];
#pragma unroll
    for (int k = 1; k < K; ++k) cm = fmaxf(cm, x[k]);
    const float nm = fmaxf(m, cm);
    const float sh = safe_shift(nm);
    float t = 0.f;
#pragma unroll
    for (int k = 0; k < K; ++k) t += fexp(x[k] - sh);
    s = s * fexp(m - sh) + t;
    m = nm;
}
__device__ __forceinline__ float lse_val(float m, float s) {
    return m == -INFINITY ? -INFINITY : m + flog(s);
}
// The same with float64 terms and maximum, for terms that are sums of float32 values of large
// magnitude (raw potentials plus message entries): a term is rounded to float32 only once the
// maximum is taken off, where it is small, so the state keeps the terms' full precision.
template <int K>
__device__ __forceinline__ void lse_fold_d(double& m, float& s, const double (&x)[K]) {
    double cm = x[0];
#pragma unroll
    for (int k = 1; k < K; ++k) cm = fmax(cm, x[k]);
    const double nm = fmax(m, cm);
    const double sh = nm == -INFINITY ? 0.0 : nm;
    float t = 0.f;
#pragma unroll
    for (int k = 0; k < K; ++k) t += fexp((float)(x[k] - sh));
    s = s * fexp((float)(m - sh)) + t;
    m = nm;
}
__device__ __forceinline__ double lse_val_d(double m, float s) {
    return m == -INFINITY ? -INFINITY : m + (double)flog(s);
}
// either fold, by the terms' type
template <int K, typename Tm>
__device__ __forceinline__ void lse_fold_t(Tm& m, float& s, const Tm (&x)[K]) {
    if constexpr (sizeof(Tm) == sizeof(double))
        lse_fold_d<K>(m, s, x);
    else
        lse_fold<K>(m, s, x);
}

// Blocks are dispatched round-robin over the 8 XCDs (block i -> XCD i % 8).  Logical block
// lid = node * ntiles + tile: the tiles of one node go to one XCD, one after another (they
// share operand strips in that XCD's L2), and consecutive nodes go to consecutive XCDs, so
// the work stays spread over all eight when only a prefix of each sequence's nodes is
// present (variable lengths).  The grid must hold node_grid(nodes, ntiles) blocks; blocks
// past the last node get lid >= nodes * ntiles.
__device__ __forceinline__ int64_t xcd_node_swizzle(int64_t bid, int ntiles) {
    const int64_t x = bid & 7, j = bid >> 3;
    const int64_t ng = j / ntiles, tile = j - ng * ntiles;
    return (ng * 8 + x) * ntiles + tile;
}
inline int64_t node_grid(int64_t nodes, int ntiles) { return (nodes + 7) / 8 * 8 * ntiles; }

}  // namespace tsc
