// Elastic implicit-GEMM kernel on MFMA for gfx950: convolution (NHWC activations,
// [Cout][KH][KW][Cin] weights), fully connected layers and strided batched
// products, with the bias / batch-norm / residual / activation epilogue fused.
//
// GEMM view: Y[m][n] = sum_k A[m][k] * B[n][k] with
//   m = output pixel (image, p, q)   n = output channel   k = (r, s, c), c fastest
//   A[m][k] = x[image, p*stride - pad + r, q*stride - pad + s, c]  (0 in the padding)
// A fully connected layer is the 1x1 case on 1x1 images (H = W = 1, row stride ldx).
//
// Logical tile = TM x TN outputs, split 2 x 2 over the 4 logical waves, each
// wave owning (TM/2) x (TN/2) outputs made of MS x MS MFMA blocks.  Operands are
// staged through LDS in K-chunks of KT with double buffering.  For every output
// element the sequence of MFMA instructions (same opcode, same K order) does not
// depend on the shard, the grid or the physical block, so results are bitwise
// identical across elastic configurations (§6.4 computational equivalence).
#pragma once

#include "elastic_common.h"

namespace miriam {

// ------------------------------------------------------------------ MFMA ops
template <class T, int MS> struct Mfma;

template <> struct Mfma<half_t, 32> {
    static constexpr int KPL = 8, NACC = 16;
    typedef f16x8 op_t;
    typedef f32x16 acc_t;
    static __device__ __forceinline__ acc_t run(op_t a, op_t b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, c, 0, 0, 0);
    }
};
template <> struct Mfma<half_t, 16> {
    static constexpr int KPL = 8, NACC = 4;
    typedef f16x8 op_t;
    typedef f32x4 acc_t;
    static __device__ __forceinline__ acc_t run(op_t a, op_t b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
};
template <> struct Mfma<bf16_t, 32> {
    static constexpr int KPL = 8, NACC = 16;
    typedef bf16x8 op_t;
    typedef f32x16 acc_t;
    static __device__ __forceinline__ acc_t run(op_t a, op_t b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
    }
};
template <> struct Mfma<bf16_t, 16> {
    static constexpr int KPL = 8, NACC = 4;
    typedef bf16x8 op_t;
    typedef f32x4 acc_t;
    static __device__ __forceinline__ acc_t run(op_t a, op_t b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
};
template <> struct Mfma<float, 32> {
    static constexpr int KPL = 1, NACC = 16;
    typedef float op_t;
    typedef f32x16 acc_t;
    static __device__ __forceinline__ acc_t run(op_t a, op_t b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
    }
};
template <> struct Mfma<float, 16> {
    static constexpr int KPL = 1, NACC = 4;
    typedef float op_t;
    typedef f32x4 acc_t;
    static __device__ __forceinline__ acc_t run(op_t a, op_t b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
};

template <class T, int TM, int TN, int MS, int P, int LAY>
struct IgemmKernel {
    typedef Mfma<T, MS> MF;
    typedef typename MF::op_t op_t;
    typedef typename MF::acc_t acc_t;
    static constexpr int NT = kWave * P;                 // physical threads
    static constexpr int VEC = 16 / (int)sizeof(T);      // elements per 16-byte vector
    static constexpr int KSTEP = (kWave / MS) * MF::KPL; // K consumed by one MFMA
    static constexpr int KT = sizeof(T) == 4 ? 32 : 64;  // K per LDS chunk
    static constexpr int PK = VEC;                       // row padding (16 bytes)
    static constexpr int LDK = KT + PK;                  // LDS row length in elements
    static constexpr int KPR = KT / VEC;                 // vectors per K-chunk row
    static constexpr int BM = TM / 2 / MS, BN = TN / 2 / MS;
    static constexpr int LW = kLogicalWaves / P;         // logical waves per physical wave
    // accumulators held at once: 128 per lane, 64 for single-wave blocks (they also hold all loads)
    static constexpr int MAXACC = P == 1 ? 64 : 128;
    static constexpr int MAXSL = (MAXACC / MF::NACC) / (BM * BN) > 0 ? (MAXACC / MF::NACC) / (BM * BN) : 1;
    static constexpr int SL = LW < MAXSL ? LW : MAXSL;   // logical waves held at once
    static constexpr int ROUNDS = LW / SL;               // sequential passes over K
    static constexpr bool A_VEC = (LAY == LAY_VEC || LAY == LAY_VEC_NB);
    static constexpr bool B_NMAJ = (LAY == LAY_VEC_NB || LAY == LAY_SCALAR_NB);
    static constexpr bool B_VEC = (LAY == LAY_VEC || LAY == LAY_VEC_NB);
    static constexpr int NVA = (TM * KPR + NT - 1) / NT;           // A vectors per thread
    static constexpr int NVB = (TN * KPR + NT - 1) / NT;           // B vectors per thread
    static constexpr int LDC = TN + 4;                   // staged output row (fp32)
    static constexpr int AB_BYTES = 2 * (TM + TN) * LDK * (int)sizeof(T);
    static constexpr int C_BYTES = TM * LDC * 4;
    static constexpr int LDS_BYTES = AB_BYTES > C_BYTES ? AB_BYTES : C_BYTES;
    static_assert(LW % SL == 0, "slots must divide logical waves");
    static_assert(KT % KSTEP == 0, "chunk must hold whole MFMA steps");
    static_assert(BM >= 1 && BN >= 1, "tile too small for the MFMA shape");
    static_assert((TN / 2) % VEC == 0, "sub-tile rows must hold whole vectors");
};

template <class T, int TM, int TN, int MS, int P, int LAY>
__global__ __launch_bounds__(kWave * P) void igemm_kernel(IgemmArgs a, Shard sh) {
    typedef IgemmKernel<T, TM, TN, MS, P, LAY> K_;
    typedef typename K_::MF MF;
    typedef typename K_::op_t op_t;
    typedef typename K_::acc_t acc_t;
    constexpr int NT = K_::NT, VEC = K_::VEC, KT = K_::KT, LDK = K_::LDK, KPR = K_::KPR;
    constexpr int BM = K_::BM, BN = K_::BN, SL = K_::SL, ROUNDS = K_::ROUNDS;
    constexpr int NVA = K_::NVA, NVB = K_::NVB, KSTEP = K_::KSTEP, LDC = K_::LDC;

    __shared__ __attribute__((aligned(16))) char smem[K_::LDS_BYTES];
    T *const lds = reinterpret_cast<T *>(smem);
    float *const Cs = reinterpret_cast<float *>(smem);
    // A tile of buffer b: rows [b*(TM+TN), +TM); B tile: the following TN rows
    auto As = [&](int b, int row) -> T * { return lds + ((b * (TM + TN)) + row) * LDK; };
    auto Bs = [&](int b, int row) -> T * { return lds + ((b * (TM + TN)) + TM + row) * LDK; };

    const int tid = threadIdx.x;
    const int pw = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int lane = tid % kWave;
    const T *__restrict__ X = static_cast<const T *>(a.x);
    const T *__restrict__ Wt = static_cast<const T *>(a.w);
    T *__restrict__ Y = static_cast<T *>(a.y);
    const T *__restrict__ R = static_cast<const T *>(a.res);
    const uint32_t HoWo32 = (uint32_t)(a.Ho * a.Wo), Wo32 = (uint32_t)a.Wo;
    const int64_t nch = (a.K + KT - 1) / KT;
    const int64_t G = gridDim.x;
    const int64_t rank = wg_rank(blockIdx.x, G);
    const int32_t C32 = (int32_t)a.C, KW32 = a.KW, KH32 = a.KH;

    int iter = 0;
    TileDigits<4> td;
    {
        const uint32_t radix[4] = {(uint32_t)a.nT, (uint32_t)a.mT, (uint32_t)a.bdiv, 0u};
        td.init((uint32_t)(sh.begin + rank), (uint32_t)G, radix);
    }
    for (int64_t t = sh.begin + rank; t < sh.begin + sh.len; t += G, ++iter, td.advance()) {
        trace_tile(sh, t, iter);
        // tile id = ((b0 * bdiv + b1) * mT + mt) * nT + nt; every index here is below 2^31
        // (checked at creation); the digits advance by the grid without division
        const uint32_t nt = td.d[0], mt = td.d[1], b1 = td.d[2], b0 = td.d[3];
        const T *Xb = X + b0 * a.sx0 + b1 * a.sx1;
        const T *Wb = Wt + b0 * a.sw0 + b1 * a.sw1;
        const int64_t yoff = b0 * a.sy0 + b1 * a.sy1;
        const int64_t m0 = (int64_t)mt * TM, n0 = (int64_t)nt * TN;

        // Per-thread A rows: image offset and the top-left input tap of the output pixel.
        int64_t a_img[NVA];
        int32_t a_h0[NVA], a_w0[NVA];
        bool a_ok[NVA];
#pragma unroll
        for (int j = 0; j < NVA; ++j) {
            const int v = tid + j * NT;
            const int row = v / KPR;
            const int64_t m = m0 + row;
            a_ok[j] = (v < TM * KPR) && (m < a.M);
            const uint32_t mm = a_ok[j] ? (uint32_t)m : 0u;
            const uint32_t img = fdiv(mm, a.fd_howo);
            const uint32_t pq = mm - img * HoWo32;
            const uint32_t p = fdiv(pq, a.fd_wo), q = pq - p * Wo32;
            a_img[j] = (int64_t)img * a.img_x;
            a_h0[j] = (int32_t)p * a.stride - a.pad;
            a_w0[j] = (int32_t)q * a.stride - a.pad;
        }

        for (int rd = 0; rd < ROUNDS; ++rd) {
            acc_t acc[SL][BM][BN];
#pragma unroll
            for (int s = 0; s < SL; ++s)
#pragma unroll
                for (int i = 0; i < BM; ++i)
#pragma unroll
                    for (int jn = 0; jn < BN; ++jn)
#pragma unroll
                        for (int e = 0; e < MF::NACC; ++e) acc[s][i][jn][e] = 0.0f;

            // (tap row, tap column, channel) of k = chunk*KT + kv*VEC for this thread's slot
            const int kv = tid % KPR;
            int32_t kr, ks, kc;
            {
                const int32_t k = kv * VEC;
                kc = k % C32;
                const int32_t tap = k / C32;
                ks = tap % KW32;
                kr = tap / KW32;
            }

            Vec16<T> ra[NVA], rb[NVB];

            auto load_chunk = [&](int64_t ch) {
                const int64_t k0 = ch * KT;
                // ---- A
#pragma unroll
                for (int j = 0; j < NVA; ++j) {
                    if constexpr (K_::A_VEC) {
                        const int32_t h = a_h0[j] + kr, w = a_w0[j] + ks;
                        const bool ok = a_ok[j] && kr < KH32 && h >= 0 && h < a.H && w >= 0 && w < a.W;
                        ra[j] = ok ? ld_vec(Xb + a_img[j] + ((int64_t)h * a.W + w) * a.ldx + kc) : zero_vec<T>();
                    } else {
                        // element loads; (r, s, c) stepped incrementally from the slot's first element
                        Vec16<T> v = zero_vec<T>();
                        int32_t r_ = kr, s_ = ks, c_ = kc;
#pragma unroll
                        for (int e = 0; e < VEC; ++e) {
                            if (a_ok[j] && r_ < KH32) {
                                const int32_t h = a_h0[j] + r_, w = a_w0[j] + s_;
                                if (h >= 0 && h < a.H && w >= 0 && w < a.W)
                                    v.e[e] = Xb[a_img[j] + ((int64_t)h * a.W + w) * a.ldx + c_];
                            }
                            if (++c_ == C32) {
                                c_ = 0;
                                if (++s_ == KW32) { s_ = 0; ++r_; }
                            }
                        }
                        ra[j] = v;
                    }
                }
                // ---- B
#pragma unroll
                for (int j = 0; j < NVB; ++j) {
                    const int v = tid + j * NT;
                    if constexpr (!K_::B_NMAJ) {
                        const int64_t n = n0 + v / KPR;
                        const int64_t k = k0 + (int64_t)kv * VEC;
                        const bool inb = v < TN * KPR && n < a.Nc;
                        if constexpr (K_::B_VEC) {
                            rb[j] = (inb && k < a.K) ? ld_vec(Wb + n * a.ldw + k) : zero_vec<T>();
                        } else {
                            Vec16<T> t2 = zero_vec<T>();
#pragma unroll
                            for (int e = 0; e < VEC; ++e)
                                if (inb && k + e < a.K) t2.e[e] = Wb[n * a.ldw + k + e];
                            rb[j] = t2;
                        }
                    } else {
                        // B stored [k][n]: vector along n at fixed k
                        constexpr int NPR = TN / VEC;  // vectors per k row
                        const int kl = v / NPR, nv = v % NPR;
                        const int64_t k = k0 + kl;
                        const int64_t n = n0 + (int64_t)nv * VEC;
                        const bool inb = v < TN * KPR && kl < KT && k < a.K;
                        if constexpr (K_::B_VEC) {
                            rb[j] = (inb && n < a.Nc) ? ld_vec(Wb + k * a.ldw + n) : zero_vec<T>();
                        } else {
                            Vec16<T> t2 = zero_vec<T>();
#pragma unroll
                            for (int e = 0; e < VEC; ++e)
                                if (inb && n + e < a.Nc) t2.e[e] = Wb[k * a.ldw + n + e];
                            rb[j] = t2;
                        }
                    }
                }
                // advance the slot's (r, s, c) by one chunk
                kc += KT;
                while (kc >= C32) {
                    kc -= C32;
                    if (++ks == KW32) { ks = 0; ++kr; }
                }
            };

            auto store_chunk = [&](int buf) {
#pragma unroll
                for (int j = 0; j < NVA; ++j) {
                    const int v = tid + j * NT;
                    if (v < TM * KPR) st_vec(As(buf, v / KPR) + (v % KPR) * VEC, ra[j]);
                }
#pragma unroll
                for (int j = 0; j < NVB; ++j) {
                    const int v = tid + j * NT;
                    if (v < TN * KPR) {
                        if constexpr (!K_::B_NMAJ) {
                            st_vec(Bs(buf, v / KPR) + (v % KPR) * VEC, rb[j]);
                        } else {
                            constexpr int NPR = TN / VEC;
                            const int kl = v / NPR, nv = v % NPR;
#pragma unroll
                            for (int e = 0; e < VEC; ++e) Bs(buf, nv * VEC + e)[kl] = rb[j].e[e];
                        }
                    }
                }
            };

            auto compute_chunk = [&](int buf) {
#pragma unroll
                for (int kk = 0; kk < KT / KSTEP; ++kk) {
                    const int kcol = kk * KSTEP + (lane / MS) * MF::KPL;
#pragma unroll
                    for (int s = 0; s < SL; ++s) {
                        const int lam = (rd * SL + s) * P + pw;
                        const int wm = lam >> 1, wn = lam & 1;
                        op_t bop[BN];
#pragma unroll
                        for (int jn = 0; jn < BN; ++jn)
                            bop[jn] = *reinterpret_cast<const op_t *>(Bs(buf, wn * (TN / 2) + jn * MS + lane % MS) + kcol);
#pragma unroll
                        for (int i = 0; i < BM; ++i) {
                            const op_t aop = *reinterpret_cast<const op_t *>(As(buf, wm * (TM / 2) + i * MS + lane % MS) + kcol);
#pragma unroll
                            for (int jn = 0; jn < BN; ++jn) acc[s][i][jn] = MF::run(aop, bop[jn], acc[s][i][jn]);
                        }
                    }
                }
            };

            load_chunk(0);
            store_chunk(0);
            __syncthreads();
            for (int64_t ch = 0; ch < nch; ++ch) {
                const bool more = ch + 1 < nch;
                if (more) load_chunk(ch + 1);
                compute_chunk((int)(ch & 1));
                if (more) store_chunk((int)((ch + 1) & 1));
                __syncthreads();
            }

            // ---- epilogue, stage 1: accumulators (+ bias, BN) -> LDS as fp32
#pragma unroll
            for (int s = 0; s < SL; ++s) {
                const int lam = (rd * SL + s) * P + pw;
                const int wm = lam >> 1, wn = lam & 1;
                trace_wave(sh, t, lam, pw, rd * SL + s);
#pragma unroll
                for (int jn = 0; jn < BN; ++jn) {
                    const int col = wn * (TN / 2) + jn * MS + lane % MS;
                    const int64_t n = n0 + col;
                    float sc, shf;
                    chan_affine(a.epi, n < a.Nc ? n : 0, sc, shf);
#pragma unroll
                    for (int i = 0; i < BM; ++i) {
                        float *const cb = Cs + (wm * (TM / 2) + i * MS + (lane / MS) * 4) * LDC + col;
#pragma unroll
                        for (int e = 0; e < MF::NACC; ++e) {
                            const int rr = (e / 4) * (4 * (kWave / MS)) + (e % 4);
                            cb[rr * LDC] = acc[s][i][jn][e] * sc + shf;
                        }
                    }
                }
            }
            __syncthreads();
            // ---- stage 2: + residual, activation, one rounding, coalesced row stores
            // (whole tile rows per store instruction when the pass holds both column halves)
            auto stage2 = [&](auto actc, auto resc) {
                constexpr int ACT = decltype(actc)::value;
                constexpr bool RES = decltype(resc)::value != 0;
                constexpr int SUBR = TM / 2, SUBC = TN / 2, CV = SUBC / VEC;
                constexpr bool FULL = (SL * P) % 2 == 0;
                constexpr int RV = FULL ? 2 * CV : CV;
                constexpr int ROWS = FULL ? (SL * P / 2) * SUBR : SL * P * SUBR;
                const int lam0 = rd * SL * P;
                for (int idx = tid; idx < ROWS * RV; idx += NT) {
                    const int rr2 = idx / RV, cv = idx - (idx / RV) * RV;
                    const int blk = rr2 / SUBR, r = rr2 - blk * SUBR;
                    const int lam = FULL ? lam0 + 2 * blk : lam0 + blk;
                    const int row = (lam >> 1) * SUBR + r;
                    const int col = FULL ? cv * VEC : (lam & 1) * SUBC + cv * VEC;
                    const int64_t m = m0 + row, n = n0 + col;
                    if (m >= a.M) continue;
                    const float *cr = Cs + row * LDC + col;
                    const int64_t off = yoff + m * a.ldy + n;
                    if (a.vec_store && n + VEC <= a.Nc) {
                        Vec16<T> o;
                        if constexpr (RES) {
                            const Vec16<T> rv = ld_vec(R + off);
#pragma unroll
                            for (int e = 0; e < VEC; ++e)
                                o.e[e] = TypeOps<T>::from_f(act_c<ACT>(cr[e] + TypeOps<T>::to_f(rv.e[e])));
                        } else {
#pragma unroll
                            for (int e = 0; e < VEC; ++e) o.e[e] = TypeOps<T>::from_f(act_c<ACT>(cr[e]));
                        }
                        st_vec(Y + off, o);
                    } else {
#pragma unroll
                        for (int e = 0; e < VEC; ++e)
                            if (n + e < a.Nc) st_f(Y + off + e, act_c<ACT>(RES ? cr[e] + ld_f(R + off + e) : cr[e]));
                    }
                }
            };
            if (a.epi.flags & EPI_RES) with_act(a.epi.act, [&](auto actc) { stage2(actc, ActTag<1>{}); });
            else with_act(a.epi.act, [&](auto actc) { stage2(actc, ActTag<0>{}); });
            __syncthreads();
        }
    }
}

// Host-side launcher for one (dtype, tile config, physical block, layout).
template <class T, int TM, int TN, int MS, int P, int LAY>
hipError_t igemm_launch(const IgemmArgs &a, const Shard &sh, int grid, hipStream_t st) {
    hipLaunchKernelGGL((igemm_kernel<T, TM, TN, MS, P, LAY>), dim3(grid), dim3(kWave * P), 0, st, a, sh);
    return hipGetLastError();
}

}  // namespace miriam

namespace miriam {

template <class T, int TM, int TN, int MS, int LAY>
inline void igemm_table(const void *out[3], int *lds) {
    out[0] = reinterpret_cast<const void *>(&igemm_kernel<T, TM, TN, MS, 1, LAY>);
    out[1] = reinterpret_cast<const void *>(&igemm_kernel<T, TM, TN, MS, 2, LAY>);
    out[2] = reinterpret_cast<const void *>(&igemm_kernel<T, TM, TN, MS, 4, LAY>);
    *lds = IgemmKernel<T, TM, TN, MS, 4, LAY>::LDS_BYTES;
}

template <class T, int LAY>
inline int igemm_table_cfg(int cfg, const void *out[3], int *lds) {
    switch (cfg) {
    case CFG_32: igemm_table<T, 32, 32, 16, LAY>(out, lds); return 0;
    case CFG_64: igemm_table<T, 64, 64, 32, LAY>(out, lds); return 0;
    case CFG_128: igemm_table<T, 128, 128, 32, LAY>(out, lds); return 0;
    case CFG_128x64: igemm_table<T, 128, 64, 32, LAY>(out, lds); return 0;
    case CFG_256x128: igemm_table<T, 256, 128, 32, LAY>(out, lds); return 0;
    default: return -1;
    }
}

}  // namespace miriam
