// Direct 3x3 / stride-1 convolution with the weights resident in registers, for
// narrow layers (C <= 64 input channels, at most 64 output channels, fp16 / bf16).
//
// The tile is the one of the direct 3x3 kernel: 4 x 32 output pixels of one image
// times 64 output channels (so the tile space, the shard plans and the tile map are
// the same), split 2 x 2 over the 4 logical waves; logical wave (wm, wn) owns tile rows
// 2wm, 2wm+1 and output channels 32wn .. 32wn+31.
//
// With at most 64 input channels the whole filter slice of a logical wave, 32
// channels x 9C K values, fits its registers as MFMA B operands (9C/4 VGPRs: 144 for
// C = 64), so a workgroup loads its weights once and keeps them across every tile it
// runs.  Only the input patch of a tile, the (4+2) x (32+2) pixels its nine taps touch,
// streams through LDS: it is DMA'd (global_load_lds_dwordx4) into one of two buffers
// while the previous tile computes.  A pixel occupies C/8 16-byte slots plus, for
// C >= 16, one padding slot, so 32 consecutive pixels of a tap map to distinct bank
// groups and every MFMA operand read is a ds_read_b128 with a compile-time offset.
//
// K order per output element (fixed, whatever the elastic configuration): MFMA step s
// covers k = 16s .. 16s+15 with k = tap * C + c (tap = 3r + s in row-major order, c
// fastest), the order of the [Cout][KH][KW][Cin] weight rows; when 9C is not a multiple
// of 16 (C = 8) the last step's upper half is zero on both operands.
//
// Elastic block: a physical block of P waves runs logical wave lambda on wave
// lambda mod P.  P = 2 runs both row halves of one channel half (same weights) at once;
// P = 1 runs the channel halves in two rounds, reloading the weights per round.  Each
// output element sees the same MFMA sequence in every configuration, so results are
// bit-identical for every shard plan, grid and physical block.
#pragma once

#include "igemm_dma.h"

namespace miriam {

template <class T, int C, int P>
struct RwKernel {
    typedef Mfma<T, 32> MF;
    static_assert(sizeof(T) == 2, "16-bit operands only");
    static_assert(C == 8 || C == 16 || C == 32 || C == 64, "C must be 8, 16, 32 or 64");
    static constexpr int TH = 4, TW = 32, TM = TH * TW, TN = 64;
    static constexpr int NT = kWave * P;
    static constexpr int VEC = 8;                         // 16-bit elements per 16 bytes
    static constexpr int NP = C / 8;                      // 16-byte pieces of a pixel
    static constexpr int SP = NP == 1 ? 1 : NP + 1;       // LDS slots per pixel (odd stride)
    static constexpr int PS = SP * 16;                    // LDS bytes per patch pixel
    static constexpr int PH = TH + 2, PW = TW + 2, PPIX = PH * PW;
    static constexpr int NSLOT = PPIX * SP;
    static constexpr int NINS = (NSLOT + kWave - 1) / kWave;  // DMA instructions per patch
    static constexpr int NJ = (NINS + P - 1) / P;             // per wave (the last may be idle)
    static constexpr int PATCH = NINS * kWave * 16;
    static constexpr int KTOT = 9 * C;
    static constexpr int NS = (KTOT + 15) / 16;            // MFMA k-steps of 16
    static constexpr int LW = kLogicalWaves / P;
    static constexpr int SL = P == 4 ? 1 : 2;              // logical waves held at once
    static constexpr int ROUNDS = LW / SL;
    static constexpr int LDC = TN + 4;                     // staged fp32 row (residual epilogue)
    static constexpr int LDY = TN + 8;                     // staged output row in elements
    static constexpr int CS = TM * LDC * 4;
    // single round: the staged tile overlays the patch buffer the tile has finished with
    static constexpr bool OVERLAY = ROUNDS == 1;
    static constexpr int BUF = OVERLAY ? (PATCH > CS ? PATCH : CS) : PATCH;
    static constexpr int LDS_BYTES = 2 * BUF + (OVERLAY ? 0 : CS);
    static constexpr int WAVES_PER_SIMD = (P == 4 && 2 * (LDS_BYTES + 16) <= 160 * 1024) ? 2 : 1;
    static_assert(LW % SL == 0, "slots");
    static_assert(TM * LDY * 2 <= CS, "staged output fits the staging area");
};

// patch pixel offset of filter tap `tap` (row-major 3x3)
template <int PW>
__host__ __device__ constexpr int rw_toff(int tap) {
    return (tap / 3) * PW + tap % 3;
}

template <class T, int C, int P>
__global__ __launch_bounds__(kWave * P, (RwKernel<T, C, P>::WAVES_PER_SIMD)) void rw3x3_kernel(IgemmArgs a,
                                                                                               Shard sh) {
    typedef RwKernel<T, C, P> K_;
    typedef typename K_::MF MF;
    typedef typename MF::op_t op_t;
    typedef typename MF::acc_t acc_t;
    constexpr int TW = K_::TW, TM = K_::TM, TN = K_::TN, PW = K_::PW, PS = K_::PS, SP = K_::SP, NP = K_::NP;
    constexpr int NT = K_::NT, VEC = K_::VEC, NS = K_::NS, SL = K_::SL, ROUNDS = K_::ROUNDS;
    constexpr int LDC = K_::LDC, LDY = K_::LDY;
    constexpr int KTOT = K_::KTOT, NJ = K_::NJ, NINS = K_::NINS, BUF = K_::BUF;

    __shared__ __attribute__((aligned(1024))) char smem_[K_::LDS_BYTES];
    const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)smem_;

    const int tid = threadIdx.x;
    const int pw = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int lane = tid % kWave;
    const int hx = lane >> 5, xl = lane & 31;  // MFMA operand half, pixel column / channel
    const T *__restrict__ X = static_cast<const T *>(a.x);
    const T *__restrict__ Wt = static_cast<const T *>(a.w);
    T *__restrict__ Y = static_cast<T *>(a.y);
    const T *__restrict__ R = static_cast<const T *>(a.res);
    const T *const zsrc = reinterpret_cast<const T *>(g_zero_src);
    const int64_t G = gridDim.x;
    const int64_t rank = wg_rank(blockIdx.x, G);
    const int64_t end = sh.begin + sh.len;
    const int32_t H32 = (int32_t)a.H, W32 = (int32_t)a.W, Ho32 = (int32_t)a.Ho, Wo32 = (int32_t)a.Wo;
    const int32_t ldx32 = (int32_t)a.ldx;
    const uint32_t tX32 = (uint32_t)a.tX, tY32 = (uint32_t)a.tY;
    const bool has_res = (a.epi.flags & EPI_RES) != 0;

    int64_t t = sh.begin + rank;
    if (t >= end) return;

    // weights of channel half wn: step s holds k = 16s + 8hx .. +7 of output channel 32wn + xl
    op_t bw[NS];
    auto load_weights = [&](int wn) {
        const int64_t n = 32 * wn + xl;
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            const int k = 16 * s + 8 * hx;
            op_t v = op_t{};
            if (n < a.Nc && k < KTOT) v = *reinterpret_cast<const op_t *>(Wt + n * a.ldw + k);
            bw[s] = v;
        }
    };
    // P = 4: logical wave pw; P = 2: channel half pw, both row halves; P = 1: both, in rounds
    if constexpr (P != 1) load_weights(P == 4 ? (pw & 1) : pw);

    // per-channel affine part of the epilogue folded into one multiply-add, v = acc * sc + sh,
    // for this lane's channel in each round (bias, then batch norm)
    float esc[ROUNDS], esh[ROUNDS];
#pragma unroll
    for (int rd = 0; rd < ROUNDS; ++rd) {
        const int wn = P == 4 ? (pw & 1) : (P == 2 ? pw : rd);
        const int64_t col = 32 * wn + xl;
        chan_affine(a.epi, col < a.Nc ? col : 0, esc[rd], esh[rd]);
    }

    // tile id = (image * tY + tile row) * tX + tile column, kept as a mixed-radix cursor that
    // advances by the grid (no division per tile)
    struct Cursor {
        uint32_t img, ty, tx;
    };
    const uint32_t gx = (uint32_t)(G % tX32), g2 = (uint32_t)(G / tX32);
    const uint32_t gy = g2 % tY32, gi = g2 / tY32;
    auto advance = [&](Cursor c) {
        c.tx += gx;
        const uint32_t cx = c.tx >= tX32 ? 1u : 0u;
        c.tx -= cx * tX32;
        c.ty += gy + cx;
        const uint32_t cy = c.ty >= tY32 ? 1u : 0u;
        c.ty -= cy * tY32;
        c.img += gi + cy;
        return c;
    };

    // DMA of the patch of tile `c` into buffer `buf`: instruction j writes slots 64j .. 64j+63
    auto issue_patch = [&](Cursor c, int buf) {
        const uint32_t tx = c.tx, ty = c.ty, img = c.img;
        const int32_t iy0 = (int32_t)ty * K_::TH - a.pad, ix0 = (int32_t)tx * TW - a.pad;
        const T *xb = X + (int64_t)img * a.img_x;
        const uint32_t base = lds0 + (uint32_t)(buf * BUF);
        // the lane index passes through an empty asm so this lane's slot decode is recomputed
        // at each call instead of being hoisted out of the tile loop, where its results would
        // sit in registers next to the resident weights
        int ln = lane;
        asm volatile("" : "+v"(ln));
#pragma unroll
        for (int jj = 0; jj < NJ; ++jj) {
            const int j = jj * P + pw;
            if (j < NINS) {
                const int q = j * kWave + ln;
                const int pr = q / SP, sl = q - (q / SP) * SP;
                const int prow = pr / PW, pcol = pr - (pr / PW) * PW;
                const int32_t iy = iy0 + prow, ix = ix0 + pcol;
                const bool ok = pr < K_::PPIX && sl < NP && (uint32_t)iy < (uint32_t)H32 && (uint32_t)ix < (uint32_t)W32;
                const int32_t off = (iy * W32 + ix) * ldx32 + sl * VEC;
                lds_dma16(ok ? xb + off : zsrc, base + (uint32_t)(j * kWave * 16));
            }
        }
    };

    Cursor cu;
    {
        const uint32_t t32 = (uint32_t)t, r2 = t32 / tX32;
        cu = Cursor{r2 / tY32, r2 % tY32, t32 % tX32};
    }
    issue_patch(cu, 0);
    int iter = 0;
    for (; t < end; t += G, ++iter) {
        trace_tile(sh, t, iter);
        const int cur = iter & 1;
        // the patch of this tile (and, on the first tile, the weights) has landed; every wave
        // is done with the other buffer (the previous tile's staged outputs)
        wait_vmcnt<0>();
        __syncthreads();
        const Cursor nx = advance(cu);
        if (t + G < end) issue_patch(nx, cur ^ 1);

        const uint32_t tx = cu.tx, ty = cu.ty, img = cu.img;
        cu = nx;
        const int32_t oy0 = (int32_t)ty * K_::TH, ox0 = (int32_t)tx * TW;
        const char *patch = smem_ + cur * BUF;
        char *const stage = smem_ + (K_::OVERLAY ? cur * BUF : 2 * BUF);
        float *const Cs = reinterpret_cast<float *>(stage);
        T *const Ys = reinterpret_cast<T *>(stage);

#pragma unroll
        for (int rd = 0; rd < ROUNDS; ++rd) {
            acc_t acc[SL][2];
            const int wn = P == 4 ? (pw & 1) : (P == 2 ? pw : rd);
            if constexpr (P == 1) load_weights(wn);
            // operand base of block i of slot sl: patch pixel (tile row y, column xl) + this lane's half
            const char *abase[SL][2];
#pragma unroll
            for (int sl = 0; sl < SL; ++sl) {
                const int wm = P == 4 ? (pw >> 1) : sl;
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    const int y = 2 * wm + i;
                    abase[sl][i] = patch + (y * PW + xl) * PS + (NP == 1 ? 0 : hx * 16);
                }
            }
            // C = 8: the two operand halves take taps 2s and 2s+1; the upper one is offset by
            // (toff(2s+1) - toff(2s)) pixels, which is 1 or PW - 2
            const int hoff1 = hx * PS, hoffw = hx * (PW - 2) * PS;
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                op_t av[SL][2];
#pragma unroll
                for (int sl = 0; sl < SL; ++sl)
#pragma unroll
                    for (int i = 0; i < 2; ++i) {
                        if constexpr (NP == 1) {
                            const int t0 = 2 * s, t1 = 2 * s + 1;
                            const int off0 = rw_toff<PW>(t0) * PS;
                            const bool wide = t1 < 9 && (rw_toff<PW>(t1) - rw_toff<PW>(t0)) != 1;
                            const char *p = abase[sl][i] + off0 + (wide ? hoffw : hoff1);
                            op_t v = *reinterpret_cast<const op_t *>(p);
                            if (16 * s + 8 * hx >= KTOT) v = op_t{};
                            av[sl][i] = v;
                        } else {
                            const int k0 = 16 * s, tap = k0 / C, c0 = k0 % C;
                            const int off = rw_toff<PW>(tap) * PS + (c0 / 8) * 16;
                            av[sl][i] = *reinterpret_cast<const op_t *>(abase[sl][i] + off);
                        }
                    }
#pragma unroll
                for (int sl = 0; sl < SL; ++sl)
#pragma unroll
                    for (int i = 0; i < 2; ++i)
                        acc[sl][i] = MF::run(av[sl][i], bw[s], s == 0 ? acc_t{} : acc[sl][i]);
            }
            // schedule: operand reads run two k-steps ahead of the MFMAs that use them
            constexpr int RD = 2 * SL;
            __builtin_amdgcn_sched_group_barrier(0x100, RD, 0);
            if constexpr (NS > 1) __builtin_amdgcn_sched_group_barrier(0x100, RD, 0);
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                __builtin_amdgcn_sched_group_barrier(0x008, RD, 0);
                if (s + 2 < NS) __builtin_amdgcn_sched_group_barrier(0x100, RD, 0);
            }
            // ---- epilogue, stage 1: v = acc * sc + sh per channel; without a residual the
            // activation and the one rounding happen here and the tile is staged in the output
            // type, otherwise it is staged as fp32 (tile row y, column x -> staged row y * TW + x)
            if constexpr (K_::OVERLAY) __syncthreads();  // every wave is done reading this patch
            const int col = 32 * wn + xl;
            auto stage1 = [&](auto actc) {
                constexpr int ACT = decltype(actc)::value;
#pragma unroll
                for (int sl = 0; sl < SL; ++sl) {
                    const int wm = P == 4 ? (pw >> 1) : sl;
#pragma unroll
                    for (int i = 0; i < 2; ++i) {
                        // element e of the block sits at tile column x = 8 (e / 4) + 4 hx + e % 4
                        const int row0 = (2 * wm + i) * TW + hx * 4;
                        float *const cb = Cs + row0 * LDC + col;
                        T *const yb = Ys + row0 * LDY + col;
#pragma unroll
                        for (int e = 0; e < MF::NACC; ++e) {
                            const int dx = (e / 4) * 8 + (e % 4);
                            const float v = acc[sl][i][e] * esc[rd] + esh[rd];
                            if constexpr (ACT < 0) cb[dx * LDC] = v;
                            else yb[dx * LDY] = TypeOps<T>::from_f(act_c<ACT>(v));
                        }
                    }
                }
            };
            if (has_res) stage1(ActTag<-1>{});
            else with_act(a.epi.act, stage1);
        }
        __syncthreads();
        // ---- stage 2: 16-byte stores of whole pixel rows (with a residual: + residual,
        // activation and the rounding first)
        constexpr int RV = TN / VEC;
        auto stage2_res = [&](auto actc) {
            constexpr int ACT = decltype(actc)::value;
#pragma unroll 1
            for (int idx = tid; idx < TM * RV; idx += NT) {
                const int row = idx / RV, cv = idx - (idx / RV) * RV;
                const int32_t oy = oy0 + row / TW, ox = ox0 + row % TW;
                const int64_t n = (int64_t)cv * VEC;
                if (oy >= Ho32 || ox >= Wo32 || n >= a.Nc) continue;
                const int64_t off = (((int64_t)img * a.Ho + oy) * a.Wo + ox) * a.ldy + n;
                const float *cr = Cs + row * LDC + cv * VEC;
                if (a.vec_store && n + VEC <= a.Nc) {
                    const Vec16<T> rv = ld_vec(R + off);
                    Vec16<T> o;
#pragma unroll
                    for (int e = 0; e < VEC; ++e) o.e[e] = TypeOps<T>::from_f(act_c<ACT>(cr[e] + TypeOps<T>::to_f(rv.e[e])));
                    st_vec(Y + off, o);
                } else {
#pragma unroll
                    for (int e = 0; e < VEC; ++e)
                        if (n + e < a.Nc) st_f(Y + off + e, act_c<ACT>(cr[e] + ld_f(R + off + e)));
                }
            }
        };
        if (has_res) {
            with_act(a.epi.act, stage2_res);
            continue;
        }
#pragma unroll 1
        for (int idx = tid; idx < TM * RV; idx += NT) {
            const int row = idx / RV, cv = idx - (idx / RV) * RV;
            const int32_t oy = oy0 + row / TW, ox = ox0 + row % TW;
            const int64_t n = (int64_t)cv * VEC;
            if (oy >= Ho32 || ox >= Wo32 || n >= a.Nc) continue;
            const int64_t off = (((int64_t)img * a.Ho + oy) * a.Wo + ox) * a.ldy + n;
            Vec16<T> o;
            {
                o.u = *reinterpret_cast<const u32x4 *>(Ys + row * LDY + cv * VEC);
                if (a.vec_store && n + VEC <= a.Nc) {
                    st_vec(Y + off, o);
                } else {
#pragma unroll
                    for (int e = 0; e < VEC; ++e)
                        if (n + e < a.Nc) Y[off + e] = o.e[e];
                }
            }
        }
    }
}

template <class T, int C>
inline void rw_table(const void *out[3], int *lds) {
    out[0] = reinterpret_cast<const void *>(&rw3x3_kernel<T, C, 1>);
    out[1] = reinterpret_cast<const void *>(&rw3x3_kernel<T, C, 2>);
    out[2] = reinterpret_cast<const void *>(&rw3x3_kernel<T, C, 4>);
    *lds = RwKernel<T, C, 4>::LDS_BYTES;
}

// Kernel table of the resident-weight kernel for C input channels; -1 if C is not served.
template <class T>
inline int rw_table_c(int64_t c, const void *out[3], int *lds) {
    switch (c) {
    case 8: rw_table<T, 8>(out, lds); return 0;
    case 16: rw_table<T, 16>(out, lds); return 0;
    case 32: rw_table<T, 32>(out, lds); return 0;
    case 64: rw_table<T, 64>(out, lds); return 0;
    default: return -1;
    }
}

}  // namespace miriam
