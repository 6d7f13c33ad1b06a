// Device-side building blocks shared by every elastic kernel of the library.
//
// Elastic grid (§6.2) + persistent threads (§6.1): a launch covers the shard
// [begin, begin+len) of an operator's logical tile space.  Physical workgroup g
// of G takes logical rank r(g) (workgroups on one die get consecutive ranks, so
// tiles that share operands share that die's L2) and runs tiles
//     t = begin + r(g) + i*G,   i = 0, 1, ...   while t < begin + len.
// Elastic block (§6.1, N:1 logical-to-physical map): the logical block is
// always 4 waves (256 threads); a physical block of P = blockDim/64 waves runs
// logical wave lambda on physical wave lambda mod P, in slot lambda div P.
// No arithmetic depends on (begin, len, G, P): each output element sees the
// same instruction sequence, so every elastic configuration is bit-identical.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "kargs.h"

namespace miriam {

typedef _Float16 half_t;
typedef __bf16 bf16_t;
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));

enum Act { ACT_NONE = 0, ACT_RELU = 1, ACT_RELU6 = 2, ACT_GELU = 3 };
enum EpiFlag { EPI_BIAS = 1, EPI_BN = 2, EPI_RES = 4 };

// n / d for n < 2^31 with the divisor's constants from make_fastdiv.
__device__ __forceinline__ uint32_t fdiv(uint32_t n, FastDiv f) {
    return (__umulhi(n, f.m) + n) >> f.s;
}

// Logical rank of physical workgroup g among G, dies dealt round-robin.
__device__ __forceinline__ int64_t wg_rank(int64_t g, int64_t G) {
    const int64_t q = G / kDies, r = G % kDies;
    const int64_t x = g % kDies, s = g / kDies;
    return x * q + (x < r ? x : r) + s;
}

__device__ __forceinline__ void trace_tile(const Shard &sh, int64_t t, int iter) {
    if (sh.count != nullptr && threadIdx.x == 0) {
        sh.owner_wg[t] = (int32_t)blockIdx.x;
        sh.owner_iter[t] = iter;
        atomicAdd(&sh.count[t], 1);
    }
}

// Record, from the physical wave that runs it, where logical wave `lam` of tile t ran:
// on physical wave `pw` of the workgroup, as the `slot`-th logical wave that wave runs.
__device__ __forceinline__ void trace_wave(const Shard &sh, int64_t t, int lam, int pw, int slot) {
    if (sh.wave_phys != nullptr && (threadIdx.x % kWave) == 0) {
        sh.wave_phys[4 * t + lam] = pw;
        sh.wave_slot[4 * t + lam] = slot;
    }
}

// ---------------------------------------------------------------- types
template <class T> struct TypeOps;
template <> struct TypeOps<float> {
    static __device__ __forceinline__ float to_f(float v) { return v; }
    static __device__ __forceinline__ float from_f(float v) { return v; }
};
template <> struct TypeOps<half_t> {
    static __device__ __forceinline__ float to_f(half_t v) { return (float)v; }
    static __device__ __forceinline__ half_t from_f(float v) { return (half_t)v; }
};
template <> struct TypeOps<bf16_t> {
    static __device__ __forceinline__ float to_f(bf16_t v) { return (float)v; }
    static __device__ __forceinline__ bf16_t from_f(float v) { return (bf16_t)v; }
};

template <class T> __device__ __forceinline__ float ld_f(const T *p) { return TypeOps<T>::to_f(*p); }
template <class T> __device__ __forceinline__ void st_f(T *p, float v) { *p = TypeOps<T>::from_f(v); }

// 16-byte vector of T: 4 floats or 8 16-bit values.
template <class T> struct Vec16 {
    static constexpr int N = 16 / (int)sizeof(T);
    union { u32x4 u; T e[16 / sizeof(T)]; };
};

template <class T> __device__ __forceinline__ Vec16<T> ld_vec(const T *p) {
    Vec16<T> v;
    v.u = *reinterpret_cast<const u32x4 *>(p);
    return v;
}
template <class T> __device__ __forceinline__ void st_vec(T *p, const Vec16<T> &v) {
    *reinterpret_cast<u32x4 *>(p) = v.u;
}
template <class T> __device__ __forceinline__ Vec16<T> zero_vec() {
    Vec16<T> v;
    v.u = u32x4{0u, 0u, 0u, 0u};
    return v;
}

// ------------------------------------------------------------- epilogue
__device__ __forceinline__ float gelu_erf(float v) {
    return 0.5f * v * (1.0f + erff(v * 0.70710678118654752440f));
}

__device__ __forceinline__ float apply_act(float v, int act) {
    switch (act) {
    case ACT_RELU: return v > 0.0f ? v : 0.0f;
    case ACT_RELU6: return fminf(fmaxf(v, 0.0f), 6.0f);
    case ACT_GELU: return gelu_erf(v);
    default: return v;
    }
}

// Activation fixed at compile time, and a dispatch that runs f(std::integral_constant<int, A>)
// once for the runtime activation, so element loops carry no per-element branch.
template <int ACT>
__device__ __forceinline__ float act_c(float v) {
    if constexpr (ACT == ACT_RELU) return v > 0.0f ? v : 0.0f;
    else if constexpr (ACT == ACT_RELU6) return fminf(fmaxf(v, 0.0f), 6.0f);
    else if constexpr (ACT == ACT_GELU) return gelu_erf(v);
    else return v;
}

template <int A>
struct ActTag {
    static constexpr int value = A;
};

template <class F>
__device__ __forceinline__ void with_act(int act, F &&f) {
    switch (act) {
    case ACT_RELU: f(ActTag<ACT_RELU>{}); break;
    case ACT_RELU6: f(ActTag<ACT_RELU6>{}); break;
    case ACT_GELU: f(ActTag<ACT_GELU>{}); break;
    default: f(ActTag<ACT_NONE>{}); break;
    }
}

// The fused epilogue  v = act(BN(acc + bias[c]) + res)  in fp32.  Split into the
// per-channel affine part (applied where the accumulator lives) and the residual /
// activation part (applied where the output is stored); same operations, same order.
struct ChanParams {
    float bias, mean, scale, beta;
};

__device__ __forceinline__ ChanParams chan_params(const Epilogue &e, int64_t c) {
    ChanParams p{0.0f, 0.0f, 1.0f, 0.0f};
    if (e.flags & EPI_BIAS) p.bias = e.bias[c];
    if (e.flags & EPI_BN) {
        p.scale = e.bn[c] / sqrtf(e.bn[3 * e.C + c] + e.eps);
        p.mean = e.bn[2 * e.C + c];
        p.beta = e.bn[e.C + c];
    }
    return p;
}

__device__ __forceinline__ float epilogue_pre(const Epilogue &e, const ChanParams &p, float acc) {
    float v = acc;
    if (e.flags & EPI_BIAS) v += p.bias;
    if (e.flags & EPI_BN) v = (v - p.mean) * p.scale + p.beta;
    return v;
}

__device__ __forceinline__ float epilogue_post(const Epilogue &e, float v, float res) {
    if (e.flags & EPI_RES) v += res;
    return apply_act(v, e.act);
}

// Per-channel affine part folded into one multiply-add, v = acc * sc + sh (bias, then batch
// norm); the residual and the activation follow.
__device__ __forceinline__ void chan_affine(const Epilogue &e, int64_t c, float &sc, float &sh) {
    const ChanParams p = chan_params(e, c);
    sc = p.scale;
    sh = (e.flags & EPI_BN) ? (p.bias - p.mean) * p.scale + p.beta : p.bias;
}

// Digits (least significant first) of a tile id in a mixed-radix tile space, advanced by a
// fixed stride with carries instead of per-tile divisions; the top digit is unbounded.
template <int L>
struct TileDigits {
    uint32_t d[L], r[L], g[L];
    __device__ __forceinline__ void init(uint32_t t, uint32_t stride, const uint32_t (&radix)[L]) {
#pragma unroll
        for (int i = 0; i + 1 < L; ++i) {
            r[i] = radix[i];
            d[i] = t % r[i];
            t /= r[i];
            g[i] = stride % r[i];
            stride /= r[i];
        }
        d[L - 1] = t;
        g[L - 1] = stride;
    }
    __device__ __forceinline__ void advance() {
        uint32_t c = 0;
#pragma unroll
        for (int i = 0; i + 1 < L; ++i) {
            const uint32_t v = d[i] + g[i] + c;  // below 2 r[i]
            c = v >= r[i] ? 1u : 0u;
            d[i] = v - c * r[i];
        }
        d[L - 1] += g[L - 1] + c;
    }
};

// Whole epilogue for one element of channel c.
__device__ __forceinline__ float epilogue_apply(const Epilogue &e, float acc, int64_t c, float res) {
    return epilogue_post(e, epilogue_pre(e, chan_params(e, c), acc), res);
}

}  // namespace miriam
