// Elastic kernels for the bandwidth-bound operators: depthwise convolution,
// max / average pooling, the standalone bias+BN+residual+activation epilogue,
// row softmax and row layer normalisation.
//
// Layout work for HBM: NHWC activations with channels fastest, so consecutive
// lanes of a wave read consecutive 16-byte channel vectors of one pixel and
// every wave access is a fully coalesced run.  Reductions (softmax, layer norm)
// give one row to one logical wave and combine lanes with a fixed xor-butterfly,
// so no LDS and no atomics are needed and the result does not depend on the
// physical block.
//
// Tiles: the logical block is 4 logical waves x 64 lanes.  Channel-vector
// kernels cover 256 "lane items" (one pixel x V channels each) per tile; row
// kernels cover 4 rows per tile.
#pragma once

#include "elastic_common.h"

namespace miriam {

// One lane item: V consecutive channels of one output pixel.
template <class T, int V, int KIND>
__device__ __forceinline__ void pix_item(const PixArgs &a, int64_t u) {
    const T *__restrict__ X = static_cast<const T *>(a.x);
    T *__restrict__ Y = static_cast<T *>(a.y);
    // item indices stay below 2^31 (checked at creation): 32-bit division
    const uint32_t CV = (uint32_t)(a.C / V), u32 = (uint32_t)u;
    const uint32_t pixu = u32 / CV;
    const int64_t pix = pixu;
    const int64_t c0 = (int64_t)(u32 - pixu * CV) * V;
    float acc[V];
    if constexpr (KIND == PIX_EW) {
        // pixel == row of C channels; elementwise epilogue
        const T *src = X + pix * a.C + c0;
        const T *rs = static_cast<const T *>(a.res) + pix * a.C + c0;
#pragma unroll
        for (int e = 0; e < V; ++e) {
            const float r = (a.epi.flags & EPI_RES) ? ld_f(rs + e) : 0.0f;
            acc[e] = epilogue_apply(a.epi, ld_f(src + e), c0 + e, r);
        }
    } else {
        const uint32_t HoWo = (uint32_t)(a.Ho * a.Wo), Wo = (uint32_t)a.Wo;
        const int64_t n = pixu / HoWo;
        const uint32_t pq = pixu - (uint32_t)n * HoWo;
        const int64_t p = pq / Wo, q = pq - (pq / Wo) * Wo;
        const int64_t h0 = p * a.stride - a.pad, w0 = q * a.stride - a.pad;
#pragma unroll
        for (int e = 0; e < V; ++e) acc[e] = (KIND == PIX_MAX) ? -INFINITY : 0.0f;
        const T *Wt = static_cast<const T *>(a.w);
        for (int r = 0; r < a.KH; ++r) {
            const int64_t h = h0 + r;
            if (h < 0 || h >= a.H) continue;
            for (int s = 0; s < a.KW; ++s) {
                const int64_t w = w0 + s;
                if (w < 0 || w >= a.W) continue;
                const T *xp = X + ((n * a.H + h) * a.W + w) * a.C + c0;
                T xv[V];
                if constexpr (V * sizeof(T) == 16) {
                    Vec16<T> vv = ld_vec(xp);
#pragma unroll
                    for (int e = 0; e < V; ++e) xv[e] = vv.e[e];
                } else {
#pragma unroll
                    for (int e = 0; e < V; ++e) xv[e] = xp[e];
                }
                if constexpr (KIND == PIX_DW) {
                    const T *wp = Wt + ((int64_t)r * a.KW + s) * a.C + c0;
                    T wv[V];
                    if constexpr (V * sizeof(T) == 16) {
                        Vec16<T> vv = ld_vec(wp);
#pragma unroll
                        for (int e = 0; e < V; ++e) wv[e] = vv.e[e];
                    } else {
#pragma unroll
                        for (int e = 0; e < V; ++e) wv[e] = wp[e];
                    }
#pragma unroll
                    for (int e = 0; e < V; ++e)
                        acc[e] = __builtin_fmaf(TypeOps<T>::to_f(xv[e]), TypeOps<T>::to_f(wv[e]), acc[e]);
                } else if constexpr (KIND == PIX_MAX) {
#pragma unroll
                    for (int e = 0; e < V; ++e) acc[e] = fmaxf(acc[e], TypeOps<T>::to_f(xv[e]));
                } else {
#pragma unroll
                    for (int e = 0; e < V; ++e) acc[e] += TypeOps<T>::to_f(xv[e]);
                }
            }
        }
        if constexpr (KIND == PIX_AVG) {
            const float inv = 1.0f / (float)(a.KH * a.KW);
#pragma unroll
            for (int e = 0; e < V; ++e) acc[e] *= inv;
        }
        if constexpr (KIND == PIX_DW) {
            const T *rs = static_cast<const T *>(a.res) + pix * a.C + c0;
#pragma unroll
            for (int e = 0; e < V; ++e) {
                const float r = (a.epi.flags & EPI_RES) ? ld_f(rs + e) : 0.0f;
                acc[e] = epilogue_apply(a.epi, acc[e], c0 + e, r);
            }
        }
    }
    T *dst = Y + pix * a.C + c0;
    if constexpr (V * sizeof(T) == 16) {
        Vec16<T> o;
#pragma unroll
        for (int e = 0; e < V; ++e) o.e[e] = TypeOps<T>::from_f(acc[e]);
        st_vec(dst, o);
    } else {
#pragma unroll
        for (int e = 0; e < V; ++e) st_f(dst + e, acc[e]);
    }
}

template <class T, int V, int KIND, int P>
__global__ __launch_bounds__(kWave * P) void pix_kernel(PixArgs a, Shard sh) {
    const int pw = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int lane = threadIdx.x % kWave;
    const int64_t G = gridDim.x;
    const int64_t rank = wg_rank(blockIdx.x, G);
    int iter = 0;
    for (int64_t t = sh.begin + rank; t < sh.begin + sh.len; t += G, ++iter) {
        trace_tile(sh, t, iter);
#pragma unroll
        for (int s = 0; s < kLogicalWaves / P; ++s) {
            const int lam = s * P + pw;
            const int64_t u = t * kLogicalBlock + lam * kWave + lane;
            if (u < a.items) pix_item<T, V, KIND>(a, u);
        }
    }
}

// ------------------------------------------------------------------- rows
__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, kWave);
    return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
    for (int off = 32; off >= 1; off >>= 1) v = fmaxf(v, __shfl_xor(v, off, kWave));
    return v;
}

// Row loads: lane handles elements j = lane*V + i*64*V (+e), in increasing i.
template <class T, int V>
__device__ __forceinline__ void ld_row_vec(const T *p, float *out) {
    if constexpr (V * sizeof(T) == 16) {
        Vec16<T> vv = ld_vec(p);
#pragma unroll
        for (int e = 0; e < V; ++e) out[e] = TypeOps<T>::to_f(vv.e[e]);
    } else {
#pragma unroll
        for (int e = 0; e < V; ++e) out[e] = ld_f(p + e);
    }
}
template <class T, int V>
__device__ __forceinline__ void st_row_vec(T *p, const float *v) {
    if constexpr (V * sizeof(T) == 16) {
        Vec16<T> o;
#pragma unroll
        for (int e = 0; e < V; ++e) o.e[e] = TypeOps<T>::from_f(v[e]);
        st_vec(p, o);
    } else {
#pragma unroll
        for (int e = 0; e < V; ++e) st_f(p + e, v[e]);
    }
}

template <class T, int V>
__device__ void softmax_row(const RowArgs &a, int64_t row, int lane) {
    const T *xr = static_cast<const T *>(a.x) + row * a.ldx;
    T *yr = static_cast<T *>(a.y) + row * a.ldy;
    float m = -INFINITY;
    for (int64_t j = (int64_t)lane * V; j < a.n; j += kWave * V) {
        float v[V];
        ld_row_vec<T, V>(xr + j, v);
#pragma unroll
        for (int e = 0; e < V; ++e) m = fmaxf(m, a.scale * v[e]);
    }
    m = wave_max(m);
    float s = 0.0f;
    for (int64_t j = (int64_t)lane * V; j < a.n; j += kWave * V) {
        float v[V];
        ld_row_vec<T, V>(xr + j, v);
#pragma unroll
        for (int e = 0; e < V; ++e) s += expf(a.scale * v[e] - m);
    }
    s = wave_sum(s);
    for (int64_t j = (int64_t)lane * V; j < a.n; j += kWave * V) {
        float v[V];
        ld_row_vec<T, V>(xr + j, v);
#pragma unroll
        for (int e = 0; e < V; ++e) v[e] = expf(a.scale * v[e] - m) / s;
        st_row_vec<T, V>(yr + j, v);
    }
}

template <class T, int V>
__device__ void layernorm_row(const RowArgs &a, int64_t row, int lane) {
    const T *xr = static_cast<const T *>(a.x) + row * a.ldx;
    const T *rr = static_cast<const T *>(a.res) + row * a.ldx;
    T *yr = static_cast<T *>(a.y) + row * a.ldy;
    auto load = [&](int64_t j, float *v) {
        ld_row_vec<T, V>(xr + j, v);
        if (a.has_res) {
            float r[V];
            ld_row_vec<T, V>(rr + j, r);
#pragma unroll
            for (int e = 0; e < V; ++e) v[e] += r[e];
        }
    };
    float s = 0.0f;
    for (int64_t j = (int64_t)lane * V; j < a.n; j += kWave * V) {
        float v[V];
        load(j, v);
#pragma unroll
        for (int e = 0; e < V; ++e) s += v[e];
    }
    const float mean = wave_sum(s) / (float)a.n;
    float q = 0.0f;
    for (int64_t j = (int64_t)lane * V; j < a.n; j += kWave * V) {
        float v[V];
        load(j, v);
#pragma unroll
        for (int e = 0; e < V; ++e) q += (v[e] - mean) * (v[e] - mean);
    }
    const float var = wave_sum(q) / (float)a.n;
    const float rstd = 1.0f / sqrtf(var + a.eps);
    for (int64_t j = (int64_t)lane * V; j < a.n; j += kWave * V) {
        float v[V];
        load(j, v);
#pragma unroll
        for (int e = 0; e < V; ++e) v[e] = (v[e] - mean) * rstd * a.gamma[j + e] + a.beta[j + e];
        st_row_vec<T, V>(yr + j, v);
    }
}

template <class T, int V, int KIND, int P>
__global__ __launch_bounds__(kWave * P) void row_kernel(RowArgs a, Shard sh) {
    const int pw = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int lane = threadIdx.x % kWave;
    const int64_t G = gridDim.x;
    const int64_t rank = wg_rank(blockIdx.x, G);
    int iter = 0;
    for (int64_t t = sh.begin + rank; t < sh.begin + sh.len; t += G, ++iter) {
        trace_tile(sh, t, iter);
        for (int s = 0; s < kLogicalWaves / P; ++s) {
            const int64_t row = t * kLogicalWaves + s * P + pw;
            if (row >= a.rows) continue;
            if constexpr (KIND == ROW_SOFTMAX) softmax_row<T, V>(a, row, lane);
            else layernorm_row<T, V>(a, row, lane);
        }
    }
}

}  // namespace miriam
