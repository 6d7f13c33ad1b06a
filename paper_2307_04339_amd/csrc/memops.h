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

// 16-byte zero source for window taps that fall in the padding.
static __device__ __attribute__((aligned(64))) uint32_t g_pix_zero[16];

// Per-channel epilogue parameters of V consecutive channels c0.. (16-byte loads when V is a
// multiple of 4: C and c0 are then multiples of 4 and the parameter rows 16-byte aligned,
// checked at creation).  Same values as chan_params, channel by channel.
template <int V>
__device__ __forceinline__ void chan_params_vec(const Epilogue &e, int64_t c0, ChanParams (&p)[V]) {
    if constexpr (V % 4 == 0) {
#pragma unroll
        for (int q = 0; q < V / 4; ++q) {
            const int64_t c = c0 + 4 * q;
            f32x4 b = {0.0f, 0.0f, 0.0f, 0.0f}, g = {1.0f, 1.0f, 1.0f, 1.0f};
            f32x4 be = {0.0f, 0.0f, 0.0f, 0.0f}, mu = {0.0f, 0.0f, 0.0f, 0.0f}, var = {0.0f, 0.0f, 0.0f, 0.0f};
            if (e.flags & EPI_BIAS) b = *reinterpret_cast<const f32x4 *>(e.bias + c);
            if (e.flags & EPI_BN) {
                g = *reinterpret_cast<const f32x4 *>(e.bn + c);
                be = *reinterpret_cast<const f32x4 *>(e.bn + e.C + c);
                mu = *reinterpret_cast<const f32x4 *>(e.bn + 2 * e.C + c);
                var = *reinterpret_cast<const f32x4 *>(e.bn + 3 * e.C + c);
            }
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                p[4 * q + i] = ChanParams{0.0f, 0.0f, 1.0f, 0.0f};
                if (e.flags & EPI_BIAS) p[4 * q + i].bias = b[i];
                if (e.flags & EPI_BN) {
                    p[4 * q + i].scale = g[i] * __builtin_amdgcn_rsqf(var[i] + e.eps);
                    p[4 * q + i].mean = mu[i];
                    p[4 * q + i].beta = be[i];
                }
            }
        }
    } else {
#pragma unroll
        for (int i = 0; i < V; ++i) p[i] = chan_params(e, c0 + i);
    }
}

template <class T, int V>
__device__ __forceinline__ void ld_items(const T *p, T (&v)[V]) {
    if constexpr (V * sizeof(T) == 16) {
        Vec16<T> vv = ld_vec(p);
#pragma unroll
        for (int e = 0; e < V; ++e) v[e] = vv.e[e];
    } else {
#pragma unroll
        for (int e = 0; e < V; ++e) v[e] = p[e];
    }
}

// One lane item: V consecutive channels of one output pixel.
// Window taps are visited in row-major order (r, then s); padding taps are skipped.  The
// taps go in batches of 9 whose loads are all issued before any is used, so a 3x3 window
// costs one round of load latency, not nine.
template <class T, int V, int KIND, int ACT>
__device__ __forceinline__ void pix_item(const PixArgs &a, int64_t u) {
    const T *__restrict__ X = static_cast<const T *>(a.x);
    T *__restrict__ Y = static_cast<T *>(a.y);
    const T *const zsrc = reinterpret_cast<const T *>(g_pix_zero);
    // item indices stay below 2^31 (checked at creation): division by precomputed constants
    const uint32_t CV = (uint32_t)(a.C / V), u32 = (uint32_t)u;
    const uint32_t pixu = fdiv(u32, a.fd_cv);
    const int64_t pix = pixu;
    const int64_t c0 = (int64_t)(u32 - pixu * CV) * V;
    float acc[V];
    if constexpr (KIND == PIX_EW) {
        // pixel == row of C channels; elementwise epilogue
        T xv[V], rv[V];
        ld_items<T, V>(X + pix * a.C + c0, xv);
        if (a.epi.flags & EPI_RES) ld_items<T, V>(static_cast<const T *>(a.res) + pix * a.C + c0, rv);
        ChanParams cp[V];
        chan_params_vec<V>(a.epi, c0, cp);
#pragma unroll
        for (int e = 0; e < V; ++e) {
            float v = epilogue_pre(a.epi, cp[e], TypeOps<T>::to_f(xv[e]));
            if (a.epi.flags & EPI_RES) v += TypeOps<T>::to_f(rv[e]);
            acc[e] = act_c<ACT>(v);
        }
    } else {
        const uint32_t HoWo = (uint32_t)(a.Ho * a.Wo), Wo = (uint32_t)a.Wo;
        const uint32_t n = fdiv(pixu, a.fd_howo);
        const uint32_t pq = pixu - n * HoWo;
        const uint32_t pu = fdiv(pq, a.fd_wo);
        const int32_t p = (int32_t)pu, q = (int32_t)(pq - pu * Wo);
        const int32_t h0 = p * a.stride - a.pad, w0 = q * a.stride - a.pad;
        const int32_t H32 = (int32_t)a.H, W32 = (int32_t)a.W;
        const int taps = a.KH * a.KW;
#pragma unroll
        for (int e = 0; e < V; ++e) acc[e] = (KIND == PIX_MAX) ? -INFINITY : 0.0f;
        const T *Wt = static_cast<const T *>(a.w);
        const T *xn = X + (int64_t)n * a.H * a.W * a.C + c0;
        int r = 0, s = 0;  // (r, s) of tap k0
        constexpr int TB = 9;  // taps per batch
        for (int k0 = 0; k0 < taps; k0 += TB) {
            T xv[TB][V], wv[TB][V];
            bool ok[TB];
            int rj = r, sj = s;
#pragma unroll
            for (int j = 0; j < TB; ++j) {
                const int32_t h = h0 + rj, w = w0 + sj;
                ok[j] = k0 + j < taps && h >= 0 && h < H32 && w >= 0 && w < W32;
                ld_items<T, V>(ok[j] ? xn + ((int64_t)h * a.W + w) * a.C : zsrc, xv[j]);
                if constexpr (KIND == PIX_DW)
                    ld_items<T, V>(ok[j] ? Wt + (int64_t)(k0 + j) * a.C + c0 : zsrc, wv[j]);
                if (++sj == a.KW) {
                    sj = 0;
                    ++rj;
                }
            }
            r = rj;
            s = sj;
#pragma unroll
            for (int j = 0; j < TB; ++j) {
                if (!ok[j]) continue;
                if constexpr (KIND == PIX_DW) {
#pragma unroll
                    for (int e = 0; e < V; ++e)
                        acc[e] = __builtin_fmaf(TypeOps<T>::to_f(xv[j][e]), TypeOps<T>::to_f(wv[j][e]), acc[e]);
                } else if constexpr (KIND == PIX_MAX) {
#pragma unroll
                    for (int e = 0; e < V; ++e) acc[e] = fmaxf(acc[e], TypeOps<T>::to_f(xv[j][e]));
                } else {
#pragma unroll
                    for (int e = 0; e < V; ++e) acc[e] += TypeOps<T>::to_f(xv[j][e]);
                }
            }
        }
        if constexpr (KIND == PIX_AVG) {
            const float inv = 1.0f / (float)(a.KH * a.KW);
#pragma unroll
            for (int e = 0; e < V; ++e) acc[e] *= inv;
        }
        if constexpr (KIND == PIX_DW) {
            T rv[V];
            if (a.epi.flags & EPI_RES) ld_items<T, V>(static_cast<const T *>(a.res) + pix * a.C + c0, rv);
            ChanParams cp[V];
            chan_params_vec<V>(a.epi, c0, cp);
#pragma unroll
            for (int e = 0; e < V; ++e) {
                float v = epilogue_pre(a.epi, cp[e], acc[e]);
                if (a.epi.flags & EPI_RES) v += TypeOps<T>::to_f(rv[e]);
                acc[e] = act_c<ACT>(v);
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

// One lane item of the 3x3 depthwise strip kernel: V consecutive channels of kDwStrip
// horizontally adjacent output pixels.  The strip's window (3 rows of (kDwStrip - 1) * ST + 3
// input pixels) is loaded once, and the weights and epilogue parameters once per item; each
// output element then takes its taps in row-major order, skipping padding taps, exactly as in
// pix_item, so the results are bitwise those of the per-pixel kernel.  Window and weights stay
// packed in registers and each input vector is widened once for the outputs that use it
// (146 VGPRs, three waves per SIMD, against 240 and two with every element widened up front:
// MobileNetV2 b32's 112x112x32 and 56x56x144 layers 32.9 -> 27.3 and 34.5 -> 28.9 us).
template <class T, int V, int ACT, int ST>
__device__ __forceinline__ void pix_dw3_item(const PixArgs &a, int64_t u) {
    constexpr int NW = (kDwStrip - 1) * ST + 3;  // input pixels per window row
    static_assert(sizeof(T) == 2 && V * sizeof(T) == 16, "strip kernel: 16-byte vectors of 16-bit channels");
    const T *__restrict__ X = static_cast<const T *>(a.x);
    T *__restrict__ Y = static_cast<T *>(a.y);
    const T *const zsrc = reinterpret_cast<const T *>(g_pix_zero);
    const uint32_t CV = (uint32_t)(a.C / V), u32 = (uint32_t)u;
    const uint32_t stu = fdiv(u32, a.fd_cv);  // strip index
    const int64_t c0 = (int64_t)(u32 - stu * CV) * V;
    const uint32_t HoWs = (uint32_t)(a.Ho * a.Ws), Ws = (uint32_t)a.Ws;
    const uint32_t n = fdiv(stu, a.fd_howo);
    const uint32_t pq = stu - n * HoWs;
    const uint32_t pu = fdiv(pq, a.fd_wo);
    const int32_t p = (int32_t)pu, q0 = (int32_t)(pq - pu * Ws) * kDwStrip;
    const int32_t h0 = p * ST - a.pad, w0 = q0 * ST - a.pad;
    const int32_t H32 = (int32_t)a.H, W32 = (int32_t)a.W, Wo32 = (int32_t)a.Wo;
    const T *xn = X + (int64_t)n * a.H * a.W * a.C + c0;
    const T *Wt = static_cast<const T *>(a.w);
    // the window and the weights stay packed (two 16-bit values per register) and are widened
    // one element at a time where they are used
    u32x4 xv[3][NW], wv[9];
    bool rok[3], cok[NW];
#pragma unroll
    for (int j = 0; j < NW; ++j) cok[j] = w0 + j >= 0 && w0 + j < W32;
#pragma unroll
    for (int r = 0; r < 3; ++r) {
        const int32_t h = h0 + r;
        rok[r] = h >= 0 && h < H32;
#pragma unroll
        for (int j = 0; j < NW; ++j)
            xv[r][j] = ld_vec(rok[r] && cok[j] ? xn + ((int64_t)h * a.W + w0 + j) * a.C : zsrc).u;
    }
#pragma unroll
    for (int k = 0; k < 9; ++k) wv[k] = ld_vec(Wt + (int64_t)k * a.C + c0).u;
    auto elem = [](const u32x4 &v, int e) -> float {
        const uint32_t w = v[e >> 1];
        const uint16_t h = (uint16_t)((e & 1) ? (w >> 16) : (w & 0xffffu));
        return TypeOps<T>::to_f(__builtin_bit_cast(T, h));
    };
    // each input vector is widened once and feeds the (up to three) outputs of the strip that
    // use it; per output the taps still come in row-major order (r, then s = j - i), skipping
    // padding taps, as in the per-pixel kernel
    float acc[kDwStrip][V];
#pragma unroll
    for (int i = 0; i < kDwStrip; ++i)
#pragma unroll
        for (int e = 0; e < V; ++e) acc[i][e] = 0.0f;
#pragma unroll
    for (int r = 0; r < 3; ++r)
#pragma unroll
        for (int j = 0; j < NW; ++j) {
            if (!(rok[r] && cok[j])) continue;
            float xf[V];
#pragma unroll
            for (int e = 0; e < V; ++e) xf[e] = elem(xv[r][j], e);
#pragma unroll
            for (int i = 0; i < kDwStrip; ++i) {
                const int sd = j - i * ST;
                if (sd < 0 || sd > 2) continue;
#pragma unroll
                for (int e = 0; e < V; ++e) acc[i][e] = __builtin_fmaf(xf[e], elem(wv[3 * r + sd], e), acc[i][e]);
            }
        }
    ChanParams cp[V];
    chan_params_vec<V>(a.epi, c0, cp);
#pragma unroll
    for (int i = 0; i < kDwStrip; ++i) {
        const int32_t q = q0 + i;
        if (q >= Wo32) break;
        const int64_t pix = ((int64_t)n * a.Ho + p) * a.Wo + q;
        T rv[V];
        if (a.epi.flags & EPI_RES) ld_items<T, V>(static_cast<const T *>(a.res) + pix * a.C + c0, rv);
        float ov[V];
#pragma unroll
        for (int e = 0; e < V; ++e) {
            float v = epilogue_pre(a.epi, cp[e], acc[i][e]);
            if (a.epi.flags & EPI_RES) v += TypeOps<T>::to_f(rv[e]);
            ov[e] = act_c<ACT>(v);
        }
        T *dst = Y + pix * a.C + c0;
        Vec16<T> o;
#pragma unroll
        for (int e = 0; e < V; ++e) o.e[e] = TypeOps<T>::from_f(ov[e]);
        st_vec(dst, o);
    }
}

template <class T, int V, int KIND, int P>
__global__ __launch_bounds__(kWave * P) void pix_kernel(PixArgs a, Shard sh) {
    const int pw = __builtin_amdgcn_readfirstlane(threadIdx.x / kWave);
    const int lane = threadIdx.x % kWave;
    const int64_t G = gridDim.x;
    const int64_t rank = wg_rank(blockIdx.x, G);
    // the activation is dispatched once for the launch, not per element
    with_act(a.epi.act, [&](auto actc) {
        constexpr int ACT = decltype(actc)::value;
        int iter = 0;
        for (int64_t t = sh.begin + rank; t < sh.begin + sh.len; t += G, ++iter) {
            trace_tile(sh, t, iter);
#pragma unroll
            for (int s = 0; s < kLogicalWaves / P; ++s) {
                const int lam = s * P + pw;
                trace_wave(sh, t, lam, pw, s);
                const int64_t u = t * kLogicalBlock + lam * kWave + lane;
                if constexpr (KIND == PIX_DW3) {
                    // stride 1 only (the library's condition for the strip kernel): a stride-2
                    // path in the same kernel would size its registers for a 9-pixel window
                    if (u < a.items) pix_dw3_item<T, V, ACT, 1>(a, u);
                } else if (u < a.items) {
                    pix_item<T, V, KIND, ACT>(a, u);
                }
            }
        }
    });
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

// Rows of up to kRowRegs vectors per lane (2048 16-bit or 1024 fp32 values) are read from
// memory once and kept in registers for every pass; longer rows are read again per pass.
// Either way each lane visits its elements j = lane V + i 64 V (+ e) in increasing i, so the
// per-element operations, and the results, are the same.
constexpr int kRowRegs = 4;

template <class T, int V>
__device__ void softmax_row_regs(const RowArgs &a, int64_t row, int lane) {
    const T *xr = static_cast<const T *>(a.x) + row * a.ldx;
    T *yr = static_cast<T *>(a.y) + row * a.ldy;
    float v[kRowRegs][V];
#pragma unroll
    for (int i = 0; i < kRowRegs; ++i) {
        const int64_t j = (int64_t)lane * V + (int64_t)i * kWave * V;
        if (j < a.n) ld_row_vec<T, V>(xr + j, v[i]);
    }
    float m = -INFINITY;
#pragma unroll
    for (int i = 0; i < kRowRegs; ++i) {
        const int64_t j = (int64_t)lane * V + (int64_t)i * kWave * V;
        if (j < a.n) {
#pragma unroll
            for (int e = 0; e < V; ++e) m = fmaxf(m, a.scale * v[i][e]);
        }
    }
    m = wave_max(m);
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < kRowRegs; ++i) {
        const int64_t j = (int64_t)lane * V + (int64_t)i * kWave * V;
        if (j < a.n) {
#pragma unroll
            for (int e = 0; e < V; ++e) {
                v[i][e] = expf(a.scale * v[i][e] - m);
                s += v[i][e];
            }
        }
    }
    s = wave_sum(s);
#pragma unroll
    for (int i = 0; i < kRowRegs; ++i) {
        const int64_t j = (int64_t)lane * V + (int64_t)i * kWave * V;
        if (j < a.n) {
#pragma unroll
            for (int e = 0; e < V; ++e) v[i][e] = v[i][e] / s;
            st_row_vec<T, V>(yr + j, v[i]);
        }
    }
}

template <class T, int V>
__device__ void softmax_row(const RowArgs &a, int64_t row, int lane) {
    if (a.n <= (int64_t)kRowRegs * kWave * V) {
        softmax_row_regs<T, V>(a, row, lane);
        return;
    }
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
__device__ void layernorm_row_regs(const RowArgs &a, int64_t row, int lane) {
    const T *xr = static_cast<const T *>(a.x) + row * a.ldx;
    const T *rr = static_cast<const T *>(a.res) + row * a.ldx;
    T *yr = static_cast<T *>(a.y) + row * a.ldy;
    float v[kRowRegs][V];
#pragma unroll
    for (int i = 0; i < kRowRegs; ++i) {
        const int64_t j = (int64_t)lane * V + (int64_t)i * kWave * V;
        if (j < a.n) {
            ld_row_vec<T, V>(xr + j, v[i]);
            if (a.has_res) {
                float r[V];
                ld_row_vec<T, V>(rr + j, r);
#pragma unroll
                for (int e = 0; e < V; ++e) v[i][e] += r[e];
            }
        }
    }
    float s = 0.0f;
#pragma unroll
    for (int i = 0; i < kRowRegs; ++i) {
        const int64_t j = (int64_t)lane * V + (int64_t)i * kWave * V;
        if (j < a.n) {
#pragma unroll
            for (int e = 0; e < V; ++e) s += v[i][e];
        }
    }
    const float mean = wave_sum(s) / (float)a.n;
    float q = 0.0f;
#pragma unroll
    for (int i = 0; i < kRowRegs; ++i) {
        const int64_t j = (int64_t)lane * V + (int64_t)i * kWave * V;
        if (j < a.n) {
#pragma unroll
            for (int e = 0; e < V; ++e) q += (v[i][e] - mean) * (v[i][e] - mean);
        }
    }
    const float var = wave_sum(q) / (float)a.n;
    const float rstd = 1.0f / sqrtf(var + a.eps);
#pragma unroll
    for (int i = 0; i < kRowRegs; ++i) {
        const int64_t j = (int64_t)lane * V + (int64_t)i * kWave * V;
        if (j < a.n) {
#pragma unroll
            for (int e = 0; e < V; ++e) v[i][e] = (v[i][e] - mean) * rstd * a.gamma[j + e] + a.beta[j + e];
            st_row_vec<T, V>(yr + j, v[i]);
        }
    }
}

template <class T, int V>
__device__ void layernorm_row(const RowArgs &a, int64_t row, int lane) {
    if (a.n <= (int64_t)kRowRegs * kWave * V) {
        layernorm_row_regs<T, V>(a, row, lane);
        return;
    }
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
            const int lam = s * P + pw;
            trace_wave(sh, t, lam, pw, s);
            const int64_t row = t * kLogicalWaves + lam;
            if (row >= a.rows) continue;
            if constexpr (KIND == ROW_SOFTMAX) softmax_row<T, V>(a, row, lane);
            else layernorm_row<T, V>(a, row, lane);
        }
    }
}

}  // namespace miriam
