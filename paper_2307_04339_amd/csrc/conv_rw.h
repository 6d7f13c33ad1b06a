// Direct convolution with the weights resident in registers, for narrow layers (fp16 /
// bf16, C <= 64 input channels): 3x3 stride 1 (at most 64 output channels), 3x3 stride 2
// (8-channel images), and 1x1 stride 1 (any number of output channels).
//
// The tile is 4 x 32 output pixels of one image times 64 output channels (for 3x3 stride 1
// the tile of the LDS-patch kernel, so the tile space, the shard plans and the tile map
// are the same), split 2 x 2 over the 4 logical waves; logical wave (wm, wn) owns tile
// rows 2wm, 2wm+1 and output channels 32wn .. 32wn+31 of the tile's 64.  Tile id =
// ((image * tY + tile row) * tX + tile column) * nT + n tile.
//
// With at most 64 input channels the whole filter slice of a logical wave, 32
// channels x KS*KS*C K values, fits its registers as MFMA B operands (9C/4 VGPRs for
// 3x3: 144 for C = 64), so with one n tile a workgroup loads its weights once and keeps
// them across every tile it runs; 1x1 layers with several n tiles load the next tile's
// (C/4 VGPRs) while the current one computes.  Only the input patch of a tile, the
// ((4-1) ST + KS) x ((32-1) ST + KS) pixels its taps touch, streams through LDS: it is
// DMA'd (global_load_lds_dwordx4) into one of two buffers while the previous tile
// computes.  A pixel occupies C/8 16-byte slots, padded to an odd count, so the pixels
// of a tap map to distinct bank groups and every MFMA operand read is a ds_read_b128 with
// a compile-time offset.
//
// K order per output element (fixed, whatever the elastic configuration): MFMA step s
// covers k = 16s .. 16s+15 with k = tap * C + c (tap = KS r + s in row-major order, c
// fastest), the order of the [Cout][KH][KW][Cin] weight rows; when KS*KS*C is not a
// multiple of 16 the last step's upper half is zero on both operands.
//
// Elastic block: a physical block of P waves runs logical wave lambda on wave
// lambda mod P, as its (lambda div P)-th logical wave.  P = 2 runs both row halves of one
// channel half (same weights) at once; P = 1 runs the four logical waves in four rounds,
// loading the weights of each round's channel half.  Each
// output element sees the same MFMA sequence in every configuration, so results are
// bit-identical for every shard plan, grid and physical block.
#pragma once

#include "igemm_dma.h"

namespace miriam {

template <class T, int C, int P, int KS, int ST>
struct RwKernel {
    typedef Mfma<T, 32> MF;
    static_assert(sizeof(T) == 2, "16-bit operands only");
    static_assert(C % 8 == 0 && C >= 8 && C <= 64, "C must be a multiple of 8 up to 64");
    // two MFMA operand halves share one tap unless one tap holds a single half (C = 8)
    static_assert(KS == 1 || C == 8 || C % 16 == 0, "3x3 needs C = 8 or a multiple of 16");
    static_assert((KS == 3 && (ST == 1 || ST == 2)) || (KS == 1 && ST == 1), "3x3 stride 1 or 2, 1x1 stride 1");
    static constexpr int TH = 4, TW = 32, TM = TH * TW, TN = 64;
    static constexpr int NT = kWave * P;
    static constexpr int VEC = 8;                         // 16-bit elements per 16 bytes
    static constexpr int NP = C / 8;                      // 16-byte pieces of a pixel
    static constexpr int SP = NP % 2 == 1 ? NP : NP + 1;  // LDS slots per pixel (odd stride)
    static constexpr int PS = SP * 16;                    // LDS bytes per patch pixel
    static constexpr int PH = (TH - 1) * ST + KS, PW = (TW - 1) * ST + KS, PPIX = PH * PW;
    static constexpr int NSLOT = PPIX * SP;
    static constexpr int NINS = (NSLOT + kWave - 1) / kWave;  // DMA instructions per patch
    static constexpr int NJ = (NINS + P - 1) / P;             // per wave (the last may be idle)
    static constexpr int PATCH = NINS * kWave * 16;
    static constexpr int KTOT = KS * KS * C;
    static constexpr int NS = (KTOT + 15) / 16;            // MFMA k-steps of 16
    static constexpr int LW = kLogicalWaves / P;
    static constexpr int SL = P == 2 ? 2 : 1;              // logical waves held at once
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

// patch pixel offset of filter tap `tap` (row-major KS x KS)
template <int PW, int KS>
__host__ __device__ constexpr int rw_toff(int tap) {
    return (tap / KS) * PW + tap % KS;
}

template <class T, int C, int P, int KS, int ST>
__global__ __launch_bounds__(kWave * P, (RwKernel<T, C, P, KS, ST>::WAVES_PER_SIMD)) void rw_conv_kernel(IgemmArgs a,
                                                                                                     Shard sh) {
    typedef RwKernel<T, C, P, KS, ST> K_;
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
    const int64_t G = gridDim.x;
    const int64_t rank = wg_rank(blockIdx.x, G);
    const int64_t end = sh.begin + sh.len;
    const int32_t H32 = (int32_t)a.H, W32 = (int32_t)a.W, Ho32 = (int32_t)a.Ho, Wo32 = (int32_t)a.Wo;
    const int32_t ldx32 = (int32_t)a.ldx;
    const uint32_t tX32 = (uint32_t)a.tX, tY32 = (uint32_t)a.tY, nT32 = (uint32_t)a.nT;
    const bool has_res = (a.epi.flags & EPI_RES) != 0;

    int64_t t = sh.begin + rank;
    if (t >= end) return;

    // weights of n tile nt, channel half wn: step s holds k = 16s + 8hx .. +7 of output
    // channel 64 nt + 32 wn + xl
    op_t bw[NS];
    auto load_weights = [&](op_t *dst, uint32_t nt, int wn) {
        const int64_t n = 64 * (int64_t)nt + 32 * wn + xl;
#pragma unroll
        for (int s = 0; s < NS; ++s) {
            const int k = 16 * s + 8 * hx;
            op_t v = op_t{};
            if (n < a.Nc && k < KTOT) v = *reinterpret_cast<const op_t *>(Wt + n * a.ldw + k);
            dst[s] = v;
        }
    };
    // P = 4: logical wave pw; P = 2: channel half pw, both row halves; P = 1: both, in rounds
    const int wn_mine = P == 4 ? (pw & 1) : (P == 2 ? pw : 0);

    // tile id = ((image * tY + tile row) * tX + tile column) * nT + n tile, kept as mixed-radix
    // digits that advance by the grid (no division per tile)
    struct Cursor {
        uint32_t img, ty, tx, nt;
    };
    const uint32_t g0 = (uint32_t)G;
    const uint32_t gn = g0 % nT32, g1 = g0 / nT32;
    const uint32_t gx = g1 % tX32, g2 = g1 / tX32;
    const uint32_t gy = g2 % tY32, gi = g2 / tY32;
    auto advance = [&](Cursor c) {
        c.nt += gn;
        const uint32_t cn = c.nt >= nT32 ? 1u : 0u;
        c.nt -= cn * nT32;
        c.tx += gx + cn;
        const uint32_t cx = c.tx >= tX32 ? 1u : 0u;
        c.tx -= cx * tX32;
        c.ty += gy + cx;
        const uint32_t cy = c.ty >= tY32 ? 1u : 0u;
        c.ty -= cy * tY32;
        c.img += gi + cy;
        return c;
    };
    const bool one_nt = nT32 == 1;
    // per-channel affine part of the epilogue folded into one multiply-add, v = acc * sc + sh,
    // for this lane's channel in each round (bias, then batch norm)
    float esc[ROUNDS], esh[ROUNDS];
    auto load_affine = [&](uint32_t nt) {
#pragma unroll
        for (int rd = 0; rd < ROUNDS; ++rd) {
            const int wn = P == 1 ? (rd & 1) : wn_mine;
            const int64_t col = 64 * (int64_t)nt + 32 * wn + xl;
            chan_affine(a.epi, col < a.Nc ? col : 0, esc[rd], esh[rd]);
        }
    };

    // DMA of the patch of tile `c` into buffer `buf`: instruction j writes slots 64j .. 64j+63.
    // The slot a lane fills is the same in every tile, so its decode (patch row and column,
    // 16-byte piece, whether the slot holds data) is done once and kept packed in one register
    // per instruction: bits [0, 7) column, [7, 11) row, [11, 15) piece, bit 15 set for a data
    // slot.  Per tile a lane then only adds the tile's origin, checks the image bounds and
    // forms a 32-bit byte offset into the image (the library admits the kernel only for images
    // of less than 2^31 bytes); pixels outside the image and padding slots take an offset past
    // the buffer, which reads zeros.
    static_assert(K_::PW < 128 && K_::PH <= 16 && SP <= 16, "packed patch geometry");
    uint32_t geo[NJ];
#pragma unroll
    for (int jj = 0; jj < NJ; ++jj) {
        const int j = jj * P + pw;
        const int q = j * kWave + lane;
        const int pr = q / SP, sl = q - (q / SP) * SP;
        const int prow = pr / PW, pcol = pr - (pr / PW) * PW;
        const bool ok = j < NINS && pr < K_::PPIX && sl < NP;
        geo[jj] = ok ? ((uint32_t)pcol | ((uint32_t)prow << 7) | ((uint32_t)sl << 11) | (1u << 15)) : 0u;
    }
    const uint32_t img_bytes = (uint32_t)(a.img_x * (int64_t)sizeof(T));
    auto issue_patch = [&](Cursor c, int buf) {
        const uint32_t tx = c.tx, ty = c.ty, img = c.img;
        const int32_t iy0 = (int32_t)ty * K_::TH * ST - a.pad, ix0 = (int32_t)tx * TW * ST - a.pad;
        const rsrc_t rs = make_rsrc(X + (int64_t)img * a.img_x, img_bytes);
        const uint32_t base = lds0 + (uint32_t)(buf * BUF);
#pragma unroll
        for (int jj = 0; jj < NJ; ++jj) {
            const int j = jj * P + pw;
            if (j < NINS) {
                const uint32_t g = geo[jj];
                const int32_t iy = iy0 + (int32_t)((g >> 7) & 15u), ix = ix0 + (int32_t)(g & 127u);
                const bool ok = (g >> 15) != 0u && (uint32_t)iy < (uint32_t)H32 && (uint32_t)ix < (uint32_t)W32;
                const uint32_t off = (uint32_t)((iy * W32 + ix) * ldx32 + (int32_t)((g >> 11) & 15u) * VEC) * (uint32_t)sizeof(T);
                buf_dma16(ok ? off : kOutOfRange, rs, 0u, base + (uint32_t)(j * kWave * 16));
            }
        }
    };

    Cursor cu;
    {
        const uint32_t t32 = (uint32_t)t, r1 = t32 / nT32, r2 = r1 / tX32;
        cu = Cursor{r2 / tY32, r2 % tY32, r1 % tX32, t32 % nT32};
    }
    // one n tile: weights and per-channel constants once for the workgroup's lifetime;
    // several (1x1 only): for each tile, the next tile's weights load with its patch
    op_t bw_next[KS == 1 ? NS : 1];
    if constexpr (P != 1) load_weights(bw, cu.nt, wn_mine);
    load_affine(cu.nt);
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
        if constexpr (KS == 1 && P != 1) {
            if (!one_nt && iter > 0) {
                // the weights loaded with this tile's patch (complete: waited above)
#pragma unroll
                for (int s = 0; s < NS; ++s) bw[s] = bw_next[s];
                load_affine(cu.nt);
            }
        }
        if (t + G < end) {
            issue_patch(nx, cur ^ 1);
            if constexpr (KS == 1 && P != 1)
                if (!one_nt) load_weights(bw_next, nx.nt, wn_mine);
        }

        const uint32_t tx = cu.tx, ty = cu.ty, img = cu.img, ntile = cu.nt;
        if constexpr (P == 1)
            if (!one_nt && iter > 0) load_affine(ntile);
        cu = nx;
        const int32_t oy0 = (int32_t)ty * K_::TH, ox0 = (int32_t)tx * TW;
        const char *patch = smem_ + cur * BUF;
        char *const stage = smem_ + (K_::OVERLAY ? cur * BUF : 2 * BUF);
        float *const Cs = reinterpret_cast<float *>(stage);
        T *const Ys = reinterpret_cast<T *>(stage);

#pragma unroll
        for (int rd = 0; rd < ROUNDS; ++rd) {
            acc_t acc[SL][2];
            // logical wave lambda = (rd SL + sl) P + pw owns tile rows 2 wm, 2 wm + 1 and channel
            // half wn, with wm = lambda div 2 and wn = lambda mod 2
            const int wn = P == 1 ? (rd & 1) : wn_mine;
            if constexpr (P == 1) load_weights(bw, ntile, wn);
            // operand base of block i of slot sl: patch pixel (tile row y, column xl) + this lane's half
            const char *abase[SL][2];
#pragma unroll
            for (int sl = 0; sl < SL; ++sl) {
                const int wm = P == 4 ? (pw >> 1) : (P == 2 ? sl : (rd >> 1));
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    const int y = 2 * wm + i;
                    abase[sl][i] = patch + (y * ST * PW + xl * ST) * PS + (NP == 1 ? 0 : hx * 16);
                }
            }
            // operands of k-step s for every block; one 8-channel tap per operand half (C = 8,
            // 3x3): halves take taps 2s and 2s+1
            auto fetch = [&](int s, op_t (&av)[SL][2]) {
#pragma unroll
                for (int sl = 0; sl < SL; ++sl)
#pragma unroll
                    for (int i = 0; i < 2; ++i) {
                        if constexpr (NP == 1 && KS == 3) {
                            const int t0 = 2 * s, t1 = 2 * s + 1;
                            const int off0 = rw_toff<PW, KS>(t0) * PS;
                            const int d1 = t1 < 9 ? (rw_toff<PW, KS>(t1) - rw_toff<PW, KS>(t0)) * PS : PS;
                            op_t v = *reinterpret_cast<const op_t *>(abase[sl][i] + off0 + hx * d1);
                            if (16 * s + 8 * hx >= KTOT) v = op_t{};
                            av[sl][i] = v;
                        } else {
                            // both halves in one tap (channels c0 .. c0 + 15); 1x1: the one tap
                            const int k0 = 16 * s, tap = KS == 1 ? 0 : k0 / C, c0 = KS == 1 ? k0 : k0 % C;
                            const int off = rw_toff<PW, KS>(tap) * PS + (c0 / 8) * 16;
                            op_t v = *reinterpret_cast<const op_t *>(abase[sl][i] + off);
                            if (KTOT % 16 != 0 && 16 * s + 8 * hx >= KTOT) v = op_t{};
                            av[sl][i] = v;
                        }
                    }
            };
            // Software pipeline in program order: the operand reads of step s + LA are issued
            // before the MFMAs of step s, and a scheduling fence after each step keeps the
            // compiler from sinking the reads next to their use (it otherwise waited on every
            // read and ran each block's MFMAs as one dependent chain).  Within a step the
            // blocks' MFMAs are independent.
            constexpr int LA = SL == 1 ? 2 : 1;
            op_t opnd[LA + 1][SL][2];
#pragma unroll
            for (int s = 0; s < LA && s < NS; ++s) fetch(s, opnd[s]);
#pragma unroll
            for (int s = 0; s < NS; ++s) {
                if (s + LA < NS) fetch(s + LA, opnd[(s + LA) % (LA + 1)]);
#pragma unroll
                for (int sl = 0; sl < SL; ++sl)
#pragma unroll
                    for (int i = 0; i < 2; ++i)
                        acc[sl][i] = MF::run(opnd[s % (LA + 1)][sl][i], bw[s], s == 0 ? acc_t{} : acc[sl][i]);
                __builtin_amdgcn_sched_barrier(0);
            }
            // ---- epilogue, stage 1: v = acc * sc + sh per channel; without a residual the
            // activation and the one rounding happen here and the tile is staged in the output
            // type, otherwise it is staged as fp32 (tile row y, column x -> staged row y * TW + x)
            if constexpr (K_::OVERLAY) __syncthreads();  // every wave is done reading this patch
            const int col = 32 * wn + xl;
#pragma unroll
            for (int sl = 0; sl < SL; ++sl)
                trace_wave(sh, t, 2 * (P == 4 ? (pw >> 1) : (P == 2 ? sl : (rd >> 1))) + wn, pw, rd * SL + sl);
            auto stage1 = [&](auto actc) {
                constexpr int ACT = decltype(actc)::value;
#pragma unroll
                for (int sl = 0; sl < SL; ++sl) {
                    const int wm = P == 4 ? (pw >> 1) : (P == 2 ? sl : (rd >> 1));
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
                const int64_t n = 64 * (int64_t)ntile + (int64_t)cv * VEC;
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
        if (a.y_bytes != 0u) {
            // whole 16-byte pieces and an output of less than 2^31 bytes: buffer stores with
            // 32-bit offsets, pieces outside the output written to an offset past the buffer
            // (dropped), no branch per piece
            static_assert((TM * RV) % NT == 0 && RV == 8 && TW == 32, "stage 2 piece decode");
            const __amdgpu_buffer_rsrc_t ry = __builtin_amdgcn_make_buffer_rsrc(Y, (short)0, (int)a.y_bytes, 0x00020000);
            // (unsigned arithmetic: the offset of a piece outside the output may wrap; it is
            // replaced before use)
            const uint32_t orow0 = ((uint32_t)img * (uint32_t)Ho32 + (uint32_t)oy0) * (uint32_t)Wo32 + (uint32_t)ox0;
            const uint32_t ldyb = (uint32_t)a.ldy * (uint32_t)sizeof(T);
#pragma unroll
            for (int it = 0; it < TM * RV / NT; ++it) {
                const int idx = tid + it * NT;
                const int row = idx >> 3, cv = idx & 7;
                const int32_t oy = oy0 + (row >> 5), ox = ox0 + (row & 31);
                const uint32_t n = 64u * ntile + (uint32_t)(cv * VEC);
                const bool ok = oy < Ho32 && ox < Wo32 && n < (uint32_t)a.Nc;
                const uint32_t off = (orow0 + (uint32_t)(row >> 5) * (uint32_t)Wo32 + (uint32_t)(row & 31)) * ldyb +
                                     n * (uint32_t)sizeof(T);
                const u32x4 v = *reinterpret_cast<const u32x4 *>(Ys + row * LDY + cv * VEC);
                __builtin_amdgcn_raw_buffer_store_b128(v, ry, (int)(ok ? off : kOutOfRange), 0, 0);
            }
            continue;
        }
#pragma unroll 1
        for (int idx = tid; idx < TM * RV; idx += NT) {
            const int row = idx / RV, cv = idx - (idx / RV) * RV;
            const int32_t oy = oy0 + row / TW, ox = ox0 + row % TW;
            const int64_t n = 64 * (int64_t)ntile + (int64_t)cv * VEC;
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

template <class T, int C, int KS, int ST>
inline void rw_table(const void *out[3], int *lds) {
    out[0] = reinterpret_cast<const void *>(&rw_conv_kernel<T, C, 1, KS, ST>);
    out[1] = reinterpret_cast<const void *>(&rw_conv_kernel<T, C, 2, KS, ST>);
    out[2] = reinterpret_cast<const void *>(&rw_conv_kernel<T, C, 4, KS, ST>);
    *lds = RwKernel<T, C, 4, KS, ST>::LDS_BYTES;
}

// Kernel table of the resident-weight kernel for a (kernel size, stride, C) it serves:
// 3x3 stride 1 with C in {8, 16, 32, 64}, 3x3 stride 2 with C = 8, 1x1 with C in
// {16, 24, 32, 64}; -1 otherwise.
template <class T>
inline int rw_table_c(int64_t ks, int64_t st, int64_t c, const void *out[3], int *lds) {
    if (ks == 3 && st == 1) {
        switch (c) {
        case 8: rw_table<T, 8, 3, 1>(out, lds); return 0;
        case 16: rw_table<T, 16, 3, 1>(out, lds); return 0;
        case 32: rw_table<T, 32, 3, 1>(out, lds); return 0;
        case 64: rw_table<T, 64, 3, 1>(out, lds); return 0;
        default: return -1;
        }
    }
    if (ks == 3 && st == 2 && c == 8) {
        rw_table<T, 8, 3, 2>(out, lds);
        return 0;
    }
    if (ks == 1 && st == 1) {
        switch (c) {
        case 16: rw_table<T, 16, 1, 1>(out, lds); return 0;
        case 24: rw_table<T, 24, 1, 1>(out, lds); return 0;
        case 32: rw_table<T, 32, 1, 1>(out, lds); return 0;
        case 64: rw_table<T, 64, 1, 1>(out, lds); return 0;
        default: return -1;
        }
    }
    return -1;
}

}  // namespace miriam
