// Direct 3x3 / stride-1 convolution kernel with the input patch held in LDS.
//
// The implicit-GEMM kernels load, for every filter tap, the tile's 128 input pixels
// again, so each input pixel crosses the L2 -> LDS path nine times.  Here a tile is a
// spatial block of TH x TW output pixels (4 rows x 32 columns) times 64 output
// channels.  For each 128-byte channel chunk, the (TH+2) x (TW+2) input pixels the
// tile's nine taps touch are loaded once into LDS (zero-filled outside the image),
// and tap (r, s) reads the A operand of output pixel (y, x) from patch row
// (y + r) * (TW + 2) + (x + s).  Only the weights stream per tap.  This cuts the
// operand bytes per flop of a 3x3 layer by about 2x against the 128x64 implicit GEMM.
//
// K order per output element (fixed, whatever the elastic configuration): channel
// chunk outer, tap (r, s) in row-major order inner, channels of the chunk innermost.
//
// Pipeline: two patch buffers (chunk cc+1 is loaded while the nine taps of chunk cc
// run) and a ring of 3 weight chunks.  Loads are global_load_lds_dwordx4 with the
// same XOR-swizzled 128-byte rows as the implicit-GEMM kernel; the waits count this
// wave's outstanding loads exactly (see the step loop).  Tiles, logical waves (2x2 of
// 64 pixels x 32 channels), MFMA shape and the staged epilogue follow igemm_dma_kernel,
// so every shard plan, grid and physical block gives bit-identical output.
#pragma once

#include "igemm_dma.h"

namespace miriam {

// s_waitcnt vmcnt(n) for a wave-uniform n; n above 47 waits for everything.
template <int N = 0>
__device__ __forceinline__ void wait_vmcnt_upto(int n) {
    if constexpr (N < 48) {
        if (n == N) {
            wait_vmcnt<N>();
            return;
        }
        wait_vmcnt_upto<N + 1>(n);
    } else {
        (void)n;
        wait_vmcnt<0>();
    }
}

template <class T, int P>
struct HaloKernel {
    typedef Mfma<T, 32> MF;
    static constexpr int TH = 4, TW = 32, TM = TH * TW, TN = 64, MS = 32;
    static constexpr int NT = kWave * P;
    static constexpr int VEC = 16 / (int)sizeof(T);
    static constexpr int KT = 128 / (int)sizeof(T);        // channels per chunk (one 128-byte row)
    static constexpr int KSTEP = (kWave / MS) * MF::KPL;
    static constexpr int PH = TH + 2, PW = TW + 2;          // input patch of the nine taps
    static constexpr int PROWS = PH * PW;                   // 204 pixels
    static constexpr int PINS = 28;                         // 8 rows per load; rows >= PROWS load zeros
    static constexpr int PATCH = PINS * 8 * 128;
    static constexpr int BSTAGE = TN * 128;
    static constexpr int SB = 3;                            // weight chunks in the ring
    static constexpr int NPW = PINS / P;                    // patch loads per wave
    static constexpr int NB = TN / 8 / P;                   // weight loads per wave per step
    static constexpr int BM = TM / 2 / MS, BN = TN / 2 / MS;
    static constexpr int LW = kLogicalWaves / P;
    static constexpr int MAXACC = P == 1 ? 64 : 128;
    static constexpr int MAXSL = (MAXACC / MF::NACC) / (BM * BN);
    static constexpr int SL = LW < MAXSL ? LW : MAXSL;
    static constexpr int ROUNDS = LW / SL;
    static constexpr int LDC = TN + 4;
    static constexpr int C_BYTES = TM * LDC * 4;
    static constexpr int RING = 2 * PATCH + SB * BSTAGE;
    static constexpr int LDS_BYTES = RING > C_BYTES ? RING : C_BYTES;
    static_assert(PINS % 4 == 0 && PINS * 8 >= PROWS, "patch loads");
    static_assert(NB >= 1 && TN % (8 * P) == 0, "weight loads");
    static_assert((SB - 2) * NB + NPW < 48, "vmcnt range");
    static_assert(LW % SL == 0 && MAXSL >= 1, "slots");
    static_assert(KT % KSTEP == 0, "chunk must hold whole MFMA steps");
    static_assert(TH / 2 == BM, "a logical wave covers two tile rows");
};

template <class T, int P>
__global__ __launch_bounds__(kWave * P, (P == 4 ? 2 : 1)) void halo_kernel(IgemmArgs a, Shard sh) {
    typedef HaloKernel<T, P> K_;
    typedef typename K_::MF MF;
    typedef typename MF::op_t op_t;
    typedef typename MF::acc_t acc_t;
    constexpr int TH = K_::TH, TW = K_::TW, TM = K_::TM, TN = K_::TN, MS = K_::MS, PW = K_::PW;
    constexpr int NT = K_::NT, VEC = K_::VEC, KT = K_::KT, KSTEP = K_::KSTEP, SB = K_::SB;
    constexpr int NPW = K_::NPW, NB = K_::NB, BM = K_::BM, BN = K_::BN, SL = K_::SL, ROUNDS = K_::ROUNDS;
    constexpr int LDC = K_::LDC;

    __shared__ __attribute__((aligned(1024))) char smem_[K_::LDS_BYTES];
    const char *const smem = smem_;
    float *const Cs = reinterpret_cast<float *>(smem_);
    const uint32_t lds0 = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)smem_;

    const int tid = threadIdx.x;
    const int pw = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int lane = tid % kWave;
    const T *__restrict__ X = static_cast<const T *>(a.x);
    const T *__restrict__ Wt = static_cast<const T *>(a.w);
    T *__restrict__ Y = static_cast<T *>(a.y);
    const T *__restrict__ R = static_cast<const T *>(a.res);
    const T *const zsrc = reinterpret_cast<const T *>(g_zero_src);
    const int CC = (int)(a.C / KT);                        // channel chunks (C is a multiple of KT)
    const int NSTEP = 9 * CC;
    const int64_t G = gridDim.x;
    const int64_t rank = wg_rank(blockIdx.x, G);
    const int32_t H32 = (int32_t)a.H, W32 = (int32_t)a.W, Ho32 = (int32_t)a.Ho, Wo32 = (int32_t)a.Wo;
    const uint32_t nT32 = (uint32_t)a.nT, tX32 = (uint32_t)a.tX, tY32 = (uint32_t)a.tY;
    const int lrow = lane >> 3, slot = lane & 7;

    int iter = 0;
    // tile id = ((image * tY + tile row) * tX + tile column) * nT + n tile, advanced by the grid
    // without division
    TileDigits<4> td;
    {
        const uint32_t radix[4] = {nT32, tX32, tY32, 0u};
        td.init((uint32_t)(sh.begin + rank), (uint32_t)G, radix);
    }
    for (int64_t t = sh.begin + rank; t < sh.begin + sh.len; t += G, ++iter, td.advance()) {
        trace_tile(sh, t, iter);
        // tile id -> (image, tile row, tile column, n tile), n fastest; ids < 2^31 (checked at creation)
        const uint32_t nt = td.d[0], tx = td.d[1], ty = td.d[2], img = td.d[3];
        const int32_t oy0 = (int32_t)ty * TH, ox0 = (int32_t)tx * TW;
        const int64_t n0 = (int64_t)nt * TN;

        // patch load j of this wave covers patch rows 8 (j P + pw) .. +7; this lane's row and piece
        const T *pbase[NPW];
        bool pok[NPW];
#pragma unroll
        for (int j = 0; j < NPW; ++j) {
            const int pr = 8 * (j * P + pw) + lrow;
            const int py = pr / PW, px = pr - (pr / PW) * PW;
            const int32_t iy = oy0 + py - a.pad, ix = ox0 + px - a.pad;
            pok[j] = pr < K_::PROWS && iy >= 0 && iy < H32 && ix >= 0 && ix < W32;
            const int64_t off = (int64_t)img * a.img_x + ((int64_t)(pok[j] ? iy : 0) * a.W + (pok[j] ? ix : 0)) * a.ldx +
                                (slot ^ ((pr >> 1) & 7)) * VEC;
            pbase[j] = X + off;
        }
        // weight load j of this wave covers output channels n0 + 8 (j P + pw) .. +7
        const T *bbase[NB];
        bool bok[NB];
#pragma unroll
        for (int j = 0; j < NB; ++j) {
            const int row = 8 * (j * P + pw) + lrow;
            const int64_t n = n0 + row;
            bok[j] = n < a.Nc;
            bbase[j] = Wt + (bok[j] ? n : 0) * a.ldw + (slot ^ ((row >> 1) & 7)) * VEC;
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

            // loads: the patch of channel chunk cc into buffer buf, the weights of step s into ring stage st
            auto issue_patch = [&](int cc, int buf) {
                const uint32_t base = lds0 + (uint32_t)(buf * K_::PATCH);
#pragma unroll
                for (int j = 0; j < NPW; ++j)
                    lds_dma16(pok[j] ? pbase[j] + (int64_t)cc * KT : zsrc, base + (uint32_t)((8 * (j * P + pw)) * 128));
            };
            auto issue_w = [&](int s, int st) {
                const int cc = s / 9, tap = s - (s / 9) * 9;
                const int64_t koff = (int64_t)tap * a.C + (int64_t)cc * KT;
                const uint32_t base = lds0 + (uint32_t)(2 * K_::PATCH + st * K_::BSTAGE);
#pragma unroll
                for (int j = 0; j < NB; ++j)
                    lds_dma16(bok[j] ? bbase[j] + koff : zsrc, base + (uint32_t)((8 * (j * P + pw)) * 128));
            };
            auto compute = [&](int s) {
                const int cc = s / 9, tap = s - (s / 9) * 9;
                const int r = tap / 3, sx = tap - (tap / 3) * 3;
                const char *patch = smem + (cc & 1) * K_::PATCH;
                const char *wst = smem + 2 * K_::PATCH + (s % SB) * K_::BSTAGE;
                constexpr int NK = KT / KSTEP;
                op_t aop[NK][SL][BM], bop[NK][SL][BN];
#pragma unroll
                for (int kk = 0; kk < NK; ++kk) {
                    const int kcol = kk * KSTEP + (lane / MS) * MF::KPL;
                    const int piece = kcol / VEC, within = (kcol % VEC) * (int)sizeof(T);
#pragma unroll
                    for (int sl = 0; sl < SL; ++sl) {
                        const int lam = (rd * SL + sl) * P + pw;
                        const int wm = lam >> 1, wn = lam & 1;
#pragma unroll
                        for (int jn = 0; jn < BN; ++jn) {
                            const int row = wn * (TN / 2) + jn * MS + lane % MS;
                            bop[kk][sl][jn] = *reinterpret_cast<const op_t *>(
                                wst + row * 128 + ((piece ^ ((row >> 1) & 7)) * 16) + within);
                        }
#pragma unroll
                        for (int i = 0; i < BM; ++i) {
                            // output pixel (y, x) of the tile = block row, lane; its tap (r, sx) input
                            const int y = wm * BM + i, x = lane % MS;
                            const int pr = (y + r) * PW + x + sx;
                            aop[kk][sl][i] = *reinterpret_cast<const op_t *>(
                                patch + pr * 128 + ((piece ^ ((pr >> 1) & 7)) * 16) + within);
                        }
                    }
                }
#pragma unroll
                for (int kk = 0; kk < NK; ++kk)
#pragma unroll
                    for (int sl = 0; sl < SL; ++sl)
#pragma unroll
                        for (int i = 0; i < BM; ++i)
#pragma unroll
                            for (int jn = 0; jn < BN; ++jn)
                                acc[sl][i][jn] = MF::run(aop[kk][sl][i], bop[kk][sl][jn], acc[sl][i][jn]);
                constexpr int RD = SL * (BM + BN), MM = SL * BM * BN;
                __builtin_amdgcn_sched_group_barrier(0x100, RD, 0);
                if constexpr (NK > 1) __builtin_amdgcn_sched_group_barrier(0x100, RD, 0);
#pragma unroll
                for (int kk = 0; kk < NK; ++kk) {
                    __builtin_amdgcn_sched_group_barrier(0x008, MM, 0);
                    if (kk + 2 < NK) __builtin_amdgcn_sched_group_barrier(0x100, RD, 0);
                }
            };

            // Issue order of this wave's loads: patch(0), W(0), W(1), then per step s (after the
            // barrier) patch(cc+1) when s opens chunk cc, then W(s+2).  At step s the loads issued
            // after W(s) are W(s+1) (issued at step s-1) and, at tap 1 only, patch(cc+1) (issued at
            // step 9 cc, after W(9 cc + 1)).  Waiting down to that count completes W(s) and every
            // earlier load, patch(cc) included.
            issue_patch(0, 0);
#pragma unroll
            for (int st = 0; st < SB - 1; ++st)
                if (st < NSTEP) issue_w(st, st);
            for (int s = 0; s < NSTEP; ++s) {
                const int cc = s / 9, tap = s - (s / 9) * 9;
                const int ahead = (NSTEP - 1 - s) < (SB - 2) ? (NSTEP - 1 - s) : (SB - 2);
                const bool patch_after = tap >= 1 && tap <= SB - 2 && cc + 1 < CC;
                wait_vmcnt_upto(ahead * NB + (patch_after ? NPW : 0));
                __syncthreads();
                if (tap == 0 && cc + 1 < CC) issue_patch(cc + 1, (cc + 1) & 1);
                if (s + SB - 1 < NSTEP) issue_w(s + SB - 1, (s + SB - 1) % SB);
                compute(s);
            }
            __syncthreads();

            // ---- epilogue, stage 1: accumulators (+ bias, BN) -> LDS as fp32; Cs row = y * TW + x
#pragma unroll
            for (int sl = 0; sl < SL; ++sl) {
                const int lam = (rd * SL + sl) * P + pw;
                const int wm = lam >> 1, wn = lam & 1;
                trace_wave(sh, t, lam, pw, rd * SL + sl);
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
                            cb[rr * LDC] = acc[sl][i][jn][e] * sc + shf;
                        }
                    }
                }
            }
            __syncthreads();
            // ---- stage 2: + residual, activation, one rounding, 16-byte stores of whole tile rows
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
                    const int blk = rr2 / SUBR, rw = rr2 - blk * SUBR;
                    const int lam = FULL ? lam0 + 2 * blk : lam0 + blk;
                    const int row = (lam >> 1) * SUBR + rw;
                    const int col = FULL ? cv * VEC : (lam & 1) * SUBC + cv * VEC;
                    const int32_t oy = oy0 + row / TW, ox = ox0 + row % TW;
                    if (oy >= Ho32 || ox >= Wo32) continue;
                    const int64_t m = ((int64_t)img * a.Ho + oy) * a.Wo + ox, n = n0 + col;
                    const float *cr = Cs + row * LDC + col;
                    const int64_t off = m * a.ldy + n;
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

template <class T>
inline int halo_table(const void *out[3], int *lds) {
    out[0] = reinterpret_cast<const void *>(&halo_kernel<T, 1>);
    out[1] = reinterpret_cast<const void *>(&halo_kernel<T, 2>);
    out[2] = reinterpret_cast<const void *>(&halo_kernel<T, 4>);
    *lds = HaloKernel<T, 4>::LDS_BYTES;
    return 0;
}

}  // namespace miriam
