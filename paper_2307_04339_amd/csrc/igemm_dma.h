// Pipelined variant of the elastic contraction kernel for 16-byte aligned, K-major
// operands (the common case: NHWC convolutions with C a multiple of 8 elements,
// fully connected layers, attention scores).
//
// Operands go straight from global memory into LDS with global_load_lds_dwordx4
// (no register staging) through a ring of S K-chunks (S-1 chunks in flight while one
// is multiplied; S is as deep as two workgroups per CU allow).  An LDS row holds one 128-byte K-chunk of one
// tile row; its eight 16-byte pieces are stored XOR-swizzled (piece c of row r
// sits at slot c ^ ((r >> 1) & 7)), which keeps the MFMA operand reads of 32
// consecutive rows free of bank conflicts without padding (each load instruction
// writes 1024 contiguous LDS bytes).  Padded taps and out-of-range rows load from
// a zero-filled device block.
//
// UNI variant: when every K chunk lies inside one filter tap (C a multiple of the chunk,
// which includes every GEMM with K a multiple of it), all lanes of a chunk share the tap
// (kh, kw) and channel base, which live in scalar registers.  Each lane then keeps a
// source pointer that is rebuilt only when the tap changes and otherwise advances by
// one chunk (by nothing for padding lanes, which point at the zero block), so a load
// costs one 64-bit add instead of a full index decode and bounds test.
//
// The arithmetic is exactly the one of igemm_kernel: same tile, same 2x2 logical
// waves, same MFMA opcode and K order, same staged epilogue; only how operands
// reach LDS differs.  Results are therefore bit-identical for every shard plan,
// grid and physical block.
#pragma once

#include "igemm.h"

namespace miriam {

// 16-byte zero source for lanes whose element lies in the padding or past a bound.
static __device__ __attribute__((aligned(64))) uint32_t g_zero_src[16];

// One 16-byte-per-lane global -> LDS load: lane i writes LDS bytes [lds + 16 i, lds + 16 i + 16).
// Issued as inline assembly so the compiler does not treat every later LDS read as
// dependent on it (it would otherwise wait for all outstanding loads before each read,
// serialising the pipeline); the kernel orders these loads itself with wait_vmcnt and
// barriers, and no compiler-visible vector loads are in flight while they are.
// `lds` is a wave-uniform LDS byte address.
__device__ __forceinline__ void lds_dma16(const void *src, uint32_t lds_addr) {
    const uint32_t lds = __builtin_amdgcn_readfirstlane(lds_addr);
    asm volatile("s_mov_b32 m0, %1\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %0, off"
                 :
                 : "v"(src), "s"(lds)
                 : "memory", "m0");
}

// Buffer resource over `bytes` bytes from `base` (raw buffer: stride 0, 32-bit offsets in
// range [0, bytes)).  A load whose per-lane offset is at or past `bytes` returns zeros, which
// the kernels use for padding taps and rows or columns past the operand's end.
typedef int32_t rsrc_t __attribute__((ext_vector_type(4)));
__device__ __forceinline__ rsrc_t make_rsrc(const void *base, uint32_t bytes) {
    const uint64_t b = (uint64_t)(uintptr_t)base;
    rsrc_t r;
    r[0] = __builtin_amdgcn_readfirstlane((int32_t)(uint32_t)b);
    r[1] = __builtin_amdgcn_readfirstlane((int32_t)((uint32_t)(b >> 32) & 0xffffu));
    r[2] = __builtin_amdgcn_readfirstlane((int32_t)bytes);
    r[3] = 0x00020000;  // 32-bit data format, no swizzle: plain byte offsets
    return r;
}
constexpr uint32_t kOutOfRange = 0x80000000u;
// cache policy of a buffer access with agent-scope coherence (sc1): what relaxed agent-scope
// atomic loads and stores compile to, here 16 bytes wide
constexpr int kAgentCoherent = 16;  // past every buffer here (spans are < 2^31 bytes)

// One 16-byte-per-lane buffer -> LDS load: lane i reads bytes [voff + soff, + 16) of the buffer
// (zeros when voff is out of range) into LDS bytes [lds + 16 i, + 16).  Ordered like lds_dma16.
__device__ __forceinline__ void buf_dma16(uint32_t voff, rsrc_t rsrc, uint32_t soff, uint32_t lds_addr) {
    const uint32_t lds = __builtin_amdgcn_readfirstlane(lds_addr);
    const uint32_t so = __builtin_amdgcn_readfirstlane(soff);
    asm volatile("s_mov_b32 m0, %2\n\ts_nop 0\n\tbuffer_load_dwordx4 %0, %1, %3 offen lds"
                 :
                 : "v"(voff), "s"(rsrc), "s"(lds), "s"(so)
                 : "memory", "m0");
}

template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt range");
    // gfx9 s_waitcnt: vmcnt bits [3:0] and [15:14]; expcnt [6:4] and lgkmcnt [11:8] left at max
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

template <class T, int TM, int TN, int MS, int P>
struct DmaKernel {
    typedef Mfma<T, MS> MF;
    static constexpr int NT = kWave * P;
    static constexpr int VEC = 16 / (int)sizeof(T);
    static constexpr int KT = 128 / (int)sizeof(T);      // one 128-byte row per chunk
    static constexpr int KSTEP = (kWave / MS) * MF::KPL;
    static constexpr int STAGE_B = (TM + TN) * 128;      // bytes per stage
    // as many stages (2..4) as keep two workgroups within a CU's 160 KB of LDS
    static constexpr int S_FIT = (80 * 1024) / STAGE_B;
    static constexpr int S = S_FIT < 2 ? 2 : (S_FIT > 4 ? 4 : S_FIT);
    static constexpr int NIA = TM / 8 / P;               // A load instructions per wave per chunk
    static constexpr int NIB = TN / 8 / P;
    static constexpr int LPC = NIA + NIB;
    static constexpr int BM = TM / 2 / MS, BN = TN / 2 / MS;
    static constexpr int LW = kLogicalWaves / P;
    static constexpr int MAXACC = P == 1 ? 64 : 128;
    static constexpr int MAXSL = (MAXACC / MF::NACC) / (BM * BN) > 0 ? (MAXACC / MF::NACC) / (BM * BN) : 1;
    static constexpr int SL = LW < MAXSL ? LW : MAXSL;
    static constexpr int ROUNDS = LW / SL;
    static constexpr int STAGE = (TM + TN) * 128;        // bytes per stage
    static constexpr int LDC = TN + 4;
    static constexpr int C_BYTES = TM * LDC * 4;
    // Split rings: where only two joint stages fit (128 x 128), the A and B operands get rings
    // of their own in the same 80 KB, three A stages and two B stages.  The weights (B) are
    // small and stay in L2; the input rows of the taps (A) also come from memory.  An A chunk
    // is then issued two chunks ahead of its use and a B chunk one (measured on VGG-16 b8
    // fp16: conv4_x 68 -> 58.5 us, conv2_2 55.4 -> 54.0 us, same bits).
    static constexpr bool SR = S == 2 && (3 * TM + 2 * TN) * 128 <= 80 * 1024;
    static constexpr int SA = SR ? 3 : S, SB = SR ? 2 : S;   // A and B stages
    static constexpr int A_STAGE = TM * 128, B_STAGE = TN * 128;
    static constexpr int RING_BYTES = SR ? SA * A_STAGE + SB * B_STAGE : S * STAGE;
    static constexpr int LDS_BYTES = RING_BYTES > C_BYTES ? RING_BYTES : C_BYTES;
    // register budget: two resident 4-wave workgroups per CU wherever their LDS fits (the split
    // rings keep no other shared variable, so they may fill exactly half of the CU's LDS)
    static constexpr int WAVES_PER_SIMD =
        (P == 4 && 2 * (LDS_BYTES + (SR ? 0 : 16)) <= 160 * 1024) ? 2 : 1;
    static_assert(TM % (8 * P) == 0 && TN % (8 * P) == 0, "load instructions must divide evenly");
    static_assert((S - 2) * LPC < 64, "vmcnt range");
    static_assert(LW % SL == 0, "slots must divide logical waves");
    static_assert(KT % KSTEP == 0, "chunk must hold whole MFMA steps");
};

// MI: memory-based index function (output-row indices from the host-computed table a.rowtab,
// staged in LDS per tile) instead of the computation-based default.
template <class T, int TM, int TN, int MS, int P, bool UNI, bool MI = false>
__global__ __launch_bounds__(kWave * P, (DmaKernel<T, TM, TN, MS, P>::WAVES_PER_SIMD)) void igemm_dma_kernel(
    IgemmArgs a, Shard sh) {
    typedef DmaKernel<T, TM, TN, MS, P> K_;
    constexpr bool SR = K_::SR;
    typedef typename K_::MF MF;
    typedef typename MF::op_t op_t;
    typedef typename MF::acc_t acc_t;
    constexpr int NT = K_::NT, VEC = K_::VEC, KT = K_::KT, KSTEP = K_::KSTEP, S = K_::S;
    constexpr int NIA = K_::NIA, NIB = K_::NIB, LPC = K_::LPC;
    constexpr int BM = K_::BM, BN = K_::BN, SL = K_::SL, ROUNDS = K_::ROUNDS, LDC = K_::LDC;

    __shared__ __attribute__((aligned(1024))) char smem_[K_::LDS_BYTES];
    char *const smem = smem_;
    float *const Cs = reinterpret_cast<float *>(smem_);
    // LDS byte address of the ring (the DMA loads take LDS addresses, not generic pointers)
    const uint32_t lds_ring = (uint32_t)(uintptr_t)(__attribute__((address_space(3))) char *)smem_;

    const int tid = threadIdx.x;
    const int pw = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int lane = tid % kWave;
    const T *__restrict__ X = static_cast<const T *>(a.x);
    const T *__restrict__ Wt = static_cast<const T *>(a.w);
    T *__restrict__ Y = static_cast<T *>(a.y);
    // output as a buffer (used when a.y_bytes != 0: whole 16-byte pieces, span below 2^31 bytes)
    const __amdgpu_buffer_rsrc_t ry = __builtin_amdgcn_make_buffer_rsrc(Y, (short)0, (int)a.y_bytes, 0x00020000);
    const T *__restrict__ R = static_cast<const T *>(a.res);
    const T *const zsrc = reinterpret_cast<const T *>(g_zero_src);
    const uint32_t HoWo32 = (uint32_t)(a.Ho * a.Wo), Wo32 = (uint32_t)a.Wo;
    const int nch = (int)((a.K + KT - 1) / KT);
    const int64_t G = gridDim.x;
    const int64_t rank = wg_rank(blockIdx.x, G);
    const int32_t C32 = (int32_t)a.C, KW32 = a.KW, KH32 = a.KH, H32 = (int32_t)a.H, W32 = (int32_t)a.W;
    const int32_t ldx32 = (int32_t)a.ldx;
    // this lane's place in every load instruction: row offset in the 8-row group, slot
    const int lrow = lane >> 3, slot = lane & 7;

    const bool has_res = (a.epi.flags & EPI_RES) != 0;
    // tile id = (((b0 * bdiv + b1) * mT + mt) * nT + nt) * ksplit + slice; indices < 2^31 (checked
    // at creation); the digits advance by the grid without division
    TileDigits<5> td;
    {
        const uint32_t radix[5] = {(uint32_t)a.ksplit, (uint32_t)a.nT, (uint32_t)a.mT, (uint32_t)a.bdiv, 0u};
        td.init((uint32_t)(sh.begin + rank), (uint32_t)G, radix);
    }
    int iter = 0;
    for (int64_t t = sh.begin + rank; t < sh.begin + sh.len; t += G, ++iter, td.advance()) {
        trace_tile(sh, t, iter);
        const uint32_t slice = td.d[0], nt = td.d[1], mt = td.d[2], b1 = td.d[3], b0 = td.d[4];
        const uint32_t otile = ((b0 * (uint32_t)a.bdiv + b1) * (uint32_t)a.mT + mt) * (uint32_t)a.nT + nt;
        const T *Xb = X + b0 * a.sx0 + b1 * a.sx1;
        const T *Wb = Wt + b0 * a.sw0 + b1 * a.sw1;
        const int64_t yoff = b0 * a.sy0 + b1 * a.sy1;
        const int64_t m0 = (int64_t)mt * TM, n0 = (int64_t)nt * TN;

        // memory-based index function: the tile's rows of the host-computed table are staged
        // in the (A) ring's last stage, which the first DMA into it (after the main loop's
        // first barrier) only overwrites once every wave has read its entries
        const int4 *const tab =
            reinterpret_cast<const int4 *>(smem + (SR ? (K_::SA - 1) * K_::A_STAGE : (S - 1) * K_::STAGE));
        if constexpr (MI) {
            const int4 *src = reinterpret_cast<const int4 *>(a.rowtab) + m0;
            for (int r = tid; r < TM; r += NT) const_cast<int4 *>(tab)[r] = src[r];
            __syncthreads();
        }
        // A instruction j of this wave covers tile rows 8q..8q+7, q = j*P + pw
        const T *a_base[NIA];
        int32_t a_h0[NIA], a_w0[NIA];
        int32_t a_kr0[NIA], a_ks0[NIA], a_kc0[NIA];
        // UNI: element offset from Xb of tap (0, 0), channel 0 + this lane's piece (negative for
        // rows whose first tap lies in the padding)
        int32_t a_row0[NIA];
        bool a_ok[NIA];
#pragma unroll
        for (int j = 0; j < NIA; ++j) {
            const int row = 8 * (j * P + pw) + lrow;
            const int64_t m = m0 + row;
            if constexpr (MI) {
                const int4 e = tab[row];
                a_ok[j] = e.w != 0;
                a_base[j] = Xb + (int64_t)e.x * a.img_x;
                a_h0[j] = e.y;
                a_w0[j] = e.z;
            } else {
                a_ok[j] = m < a.M;
                const uint32_t mm = a_ok[j] ? (uint32_t)m : 0u;
                const uint32_t img = fdiv(mm, a.fd_howo);
                const uint32_t pq = mm - img * HoWo32;
                const uint32_t p = fdiv(pq, a.fd_wo), q = pq - p * Wo32;
                a_base[j] = Xb + (int64_t)img * a.img_x;
                a_h0[j] = (int32_t)p * a.stride - a.pad;
                a_w0[j] = (int32_t)q * a.stride - a.pad;
            }
            // logical 16-byte piece of this slot, in the slice's first chunk
            const int32_t k = (int32_t)(slice * (uint32_t)a.cps) * KT + ((slot ^ ((row >> 1) & 7)) * VEC);
            if constexpr (UNI) {
                a_row0[j] = (int32_t)((a_base[j] - Xb) + ((int64_t)a_h0[j] * a.W + a_w0[j]) * a.ldx +
                                      (slot ^ ((row >> 1) & 7)) * VEC);
            } else {
                a_kc0[j] = k % C32;
                const int32_t tap = k / C32;
                a_ks0[j] = tap % KW32;
                a_kr0[j] = tap / KW32;
            }
        }
        const T *b_base[NIB];
        int32_t b_k0[NIB];
        bool b_ok[NIB];
        uint32_t b_off[NIB];  // UNI: byte offset from Wb of this lane's piece of K chunk 0 (or out of range)
#pragma unroll
        for (int j = 0; j < NIB; ++j) {
            const int row = 8 * (j * P + pw) + lrow;
            const int64_t n = n0 + row;
            b_ok[j] = n < a.Nc;
            b_base[j] = Wb + (b_ok[j] ? n : 0) * a.ldw;
            b_k0[j] = (slot ^ ((row >> 1) & 7)) * VEC;
            b_off[j] = b_ok[j] ? (uint32_t)((n * a.ldw + b_k0[j]) * (int64_t)sizeof(T)) : kOutOfRange;
        }
        // UNI: the operands as buffers (spans below 2^31 bytes, checked at creation), so padding
        // and rows past M or N read zeros from out-of-range offsets
        rsrc_t rs_a, rs_b;
        if constexpr (UNI) {
            rs_a = make_rsrc(Xb, a.x_bytes);
            rs_b = make_rsrc(Wb, a.w_bytes);
        }

        const int c0 = (int)slice * a.cps;
        const int nsl = c0 >= nch ? 0 : ((nch - c0) < a.cps ? (nch - c0) : a.cps);  // chunks of this slice
        float *const part = a.ksplit > 1 ? a.work + (int64_t)t * (TM * TN) : nullptr;

        // ---- epilogue of round rd: stage 1, accumulators * sc + sh (bias, BN) -> LDS as fp32
        auto epilogue = [&](int rd, acc_t (&acc)[SL][BM][BN]) {
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
            // ---- stage 2: + residual, activation, one rounding, coalesced row stores.
            // When this pass holds both column halves of its rows (always for 4-wave blocks),
            // consecutive threads cover whole output rows of the tile, so every store
            // instruction writes full rows (TN * sizeof(T) contiguous bytes each) rather
            // than half rows whose other halves arrive later.
            auto stage2 = [&](auto actc, auto resc) {
                constexpr int ACT = decltype(actc)::value;
                constexpr bool RES = decltype(resc)::value != 0;
                constexpr int SUBR = TM / 2, SUBC = TN / 2, CV = SUBC / VEC;
                constexpr bool FULL = (SL * P) % 2 == 0;
                constexpr int RV = FULL ? 2 * CV : CV;  // vectors per stored row segment
                constexpr int ROWS = FULL ? (SL * P / 2) * SUBR : SL * P * SUBR;
                const int lam0 = rd * SL * P;
                for (int idx = tid; idx < ROWS * RV; idx += NT) {
                    const int rr2 = idx / RV, cv = idx - (idx / RV) * RV;
                    // FULL: row block (lam0 / 2 + rr2 / SUBR) and both halves; else sub-tile lam0 + rr2 / SUBR
                    const int blk = rr2 / SUBR, r = rr2 - blk * SUBR;
                    const int lam = FULL ? lam0 + 2 * blk : lam0 + blk;
                    const int row = (lam >> 1) * SUBR + r;
                    const int col = FULL ? cv * VEC : (lam & 1) * SUBC + cv * VEC;
                    const int64_t m = m0 + row, n = n0 + col;
                    const float *cr = Cs + row * LDC + col;
                    if (!RES && a.y_bytes != 0u) {
                        // whole 16-byte pieces and an output of less than 2^31 bytes: a buffer
                        // store with a 32-bit offset (wrapping for rows past M, which are
                        // replaced by an offset past the buffer, so the store is dropped)
                        Vec16<T> o;
#pragma unroll
                        for (int e = 0; e < VEC; ++e) o.e[e] = TypeOps<T>::from_f(act_c<ACT>(cr[e]));
                        const uint32_t off = ((uint32_t)yoff + (uint32_t)m * (uint32_t)a.ldy + (uint32_t)n) * (uint32_t)sizeof(T);
                        __builtin_amdgcn_raw_buffer_store_b128(o.u, ry, (int)(m < a.M && n < a.Nc ? off : kOutOfRange), 0, 0);
                        continue;
                    }
                    if (m >= a.M) continue;
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
            if (has_res) with_act(a.epi.act, [&](auto actc) { stage2(actc, ActTag<1>{}); });
            else with_act(a.epi.act, [&](auto actc) { stage2(actc, ActTag<0>{}); });
            __syncthreads();
        };

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

            int32_t kr[NIA], ks[NIA], kc[NIA];
            if constexpr (!UNI) {
#pragma unroll
                for (int j = 0; j < NIA; ++j) {
                    kr[j] = a_kr0[j];
                    ks[j] = a_ks0[j];
                    kc[j] = a_kc0[j];
                }
            }
            // UNI: the chunk's tap (ur, us) and channel base uc are wave-uniform
            int32_t ur = 0, us = 0, uc = 0;
            bool retap = true;
            // UNI: this tap's byte offset per A instruction, fixed across the tap's chunks (the
            // chunk's channel base goes in the uniform offset); the next B chunk's byte offset
            uint32_t voff_a[NIA];
            uint32_t kb_bytes = 0;
            if constexpr (UNI) {
                const int32_t k0 = c0 * KT, tap = k0 / C32;
                uc = k0 - tap * C32;
                ur = tap / KW32;
                us = tap - ur * KW32;
                kb_bytes = (uint32_t)k0 * (uint32_t)sizeof(T);
            }

            // LDS byte addresses of chunk ch's A and B stages
            auto a_stage = [&](int ch) -> uint32_t {
                return lds_ring + (uint32_t)(SR ? (ch % K_::SA) * K_::A_STAGE : (ch % S) * K_::STAGE);
            };
            auto b_stage = [&](int ch) -> uint32_t {
                return lds_ring + (uint32_t)(SR ? K_::SA * K_::A_STAGE + (ch % K_::SB) * K_::B_STAGE
                                                : (ch % S) * K_::STAGE + TM * 128);
            };
            // issue chunk ch of A (chunks in increasing order; all lanes issue every instruction)
            auto issue_a = [&](int ch) {
                const uint32_t stage = a_stage(ch);
                if constexpr (UNI) {
                    if (retap) {
                        const int32_t toff = (ur * W32 + us) * ldx32;
#pragma unroll
                        for (int j = 0; j < NIA; ++j) {
                            const uint32_t h = (uint32_t)(a_h0[j] + ur), w = (uint32_t)(a_w0[j] + us);
                            // bitwise &: one mask and one select, no branch per lane group
                            const bool ok = a_ok[j] & (h < (uint32_t)H32) & (w < (uint32_t)W32);
                            voff_a[j] = ok ? (uint32_t)(a_row0[j] + toff) * (uint32_t)sizeof(T) : kOutOfRange;
                        }
                        retap = false;
                    }
                    const uint32_t soff = (uint32_t)uc * (uint32_t)sizeof(T);
#pragma unroll
                    for (int j = 0; j < NIA; ++j) buf_dma16(voff_a[j], rs_a, soff, stage + (uint32_t)((8 * (j * P + pw)) * 128));
                    uc += KT;
                    if (uc == C32) {
                        uc = 0;
                        retap = true;
                        if (++us == KW32) {
                            us = 0;
                            ++ur;
                        }
                    }
                    (void)ch;
                    return;
                }
#pragma unroll
                for (int j = 0; j < NIA; ++j) {
                    const int32_t h = a_h0[j] + kr[j], w = a_w0[j] + ks[j];
                    const bool ok = a_ok[j] && kr[j] < KH32 && h >= 0 && h < H32 && w >= 0 && w < W32;
                    const T *src = ok ? a_base[j] + ((int64_t)h * a.W + w) * a.ldx + kc[j] : zsrc;
                    lds_dma16(src, stage + (uint32_t)((8 * (j * P + pw)) * 128));
                    kc[j] += KT;
                    while (kc[j] >= C32) {
                        kc[j] -= C32;
                        if (++ks[j] == KW32) { ks[j] = 0; ++kr[j]; }
                    }
                }
            };
            // issue chunk ch of B (chunks in increasing order)
            auto issue_b = [&](int ch) {
                const uint32_t stage = b_stage(ch);
                if constexpr (UNI) {
#pragma unroll
                    for (int j = 0; j < NIB; ++j) buf_dma16(b_off[j], rs_b, kb_bytes, stage + (uint32_t)((8 * (j * P + pw)) * 128));
                    kb_bytes += (uint32_t)KT * (uint32_t)sizeof(T);
                    (void)ch;
                    return;
                }
                const int64_t k0 = (int64_t)(c0 + ch) * KT;
#pragma unroll
                for (int j = 0; j < NIB; ++j) {
                    const int64_t k = k0 + b_k0[j];
                    const T *src = (b_ok[j] && k < a.K) ? b_base[j] + k : zsrc;
                    lds_dma16(src, stage + (uint32_t)((8 * (j * P + pw)) * 128));
                }
            };

            auto compute = [&](int ch) {
                const char *sta = smem + (SR ? (ch % K_::SA) * K_::A_STAGE : (ch % S) * K_::STAGE);
                const char *stb = smem + (SR ? K_::SA * K_::A_STAGE + (ch % K_::SB) * K_::B_STAGE
                                             : (ch % S) * K_::STAGE + TM * 128);
                constexpr int NK = KT / KSTEP;
                // read every operand of the chunk first, so LDS latency overlaps the MFMAs
                op_t aop[NK][SL][BM], bop[NK][SL][BN];
#pragma unroll
                for (int kk = 0; kk < NK; ++kk) {
                    const int kcol = kk * KSTEP + (lane / MS) * MF::KPL;
                    const int piece = kcol / VEC, within = (kcol % VEC) * (int)sizeof(T);
#pragma unroll
                    for (int s = 0; s < SL; ++s) {
                        const int lam = (rd * SL + s) * P + pw;
                        const int wm = lam >> 1, wn = lam & 1;
#pragma unroll
                        for (int jn = 0; jn < BN; ++jn) {
                            const int row = wn * (TN / 2) + jn * MS + lane % MS;
                            bop[kk][s][jn] = *reinterpret_cast<const op_t *>(
                                stb + row * 128 + ((piece ^ ((row >> 1) & 7)) * 16) + within);
                        }
#pragma unroll
                        for (int i = 0; i < BM; ++i) {
                            const int row = wm * (TM / 2) + i * MS + lane % MS;
                            aop[kk][s][i] = *reinterpret_cast<const op_t *>(
                                sta + row * 128 + ((piece ^ ((row >> 1) & 7)) * 16) + within);
                        }
                    }
                }
#pragma unroll
                for (int kk = 0; kk < NK; ++kk)
#pragma unroll
                    for (int s = 0; s < SL; ++s)
#pragma unroll
                        for (int i = 0; i < BM; ++i)
#pragma unroll
                            for (int jn = 0; jn < BN; ++jn)
                                acc[s][i][jn] = MF::run(aop[kk][s][i], bop[kk][s][jn], acc[s][i][jn]);
                // schedule: operand reads run two MFMA steps ahead of the MFMAs that use them
                constexpr int RD = SL * (BM + BN), MM = SL * BM * BN;
                __builtin_amdgcn_sched_group_barrier(0x100, RD, 0);
                if constexpr (NK > 1) __builtin_amdgcn_sched_group_barrier(0x100, RD, 0);
#pragma unroll
                for (int kk = 0; kk < NK; ++kk) {
                    __builtin_amdgcn_sched_group_barrier(0x008, MM, 0);
                    if (kk + 2 < NK) __builtin_amdgcn_sched_group_barrier(0x100, RD, 0);
                }
            };

            if constexpr (SR) {
                // issue order: A(0), B(0), A(1), then per chunk c (after the barrier) B(c+1), A(c+2).
                // At the top of chunk c the only load issued after B(c) is A(c+1), and A(c) was
                // issued before B(c): waiting down to A(c+1)'s instructions completes both.
                if (nsl > 0) {
                    issue_a(0);
                    issue_b(0);
                }
                if (nsl > 1) issue_a(1);
                for (int c = 0; c < nsl; ++c) {
                    if (c + 1 < nsl) wait_vmcnt<NIA>();
                    else wait_vmcnt<0>();
                    __syncthreads();
                    if (c + 1 < nsl) issue_b(c + 1);
                    if (c + 2 < nsl) issue_a(c + 2);
                    compute(c);
                }
            } else {
#pragma unroll
                for (int st = 0; st < S - 1; ++st)
                    if (st < nsl) {
                        issue_a(st);
                        issue_b(st);
                    }
                for (int c = 0; c < nsl; ++c) {
                    // chunks issued after c and still allowed in flight: c+1 .. min(c+S-2, nsl-1)
                    const int pending = (nsl - 1 - c) < (S - 2) ? (nsl - 1 - c) : (S - 2);
                    if constexpr (S - 2 >= 2) {
                        if (pending >= 2) wait_vmcnt<2 * LPC>();
                        else if (pending == 1) wait_vmcnt<LPC>();
                        else wait_vmcnt<0>();
                    } else if constexpr (S - 2 == 1) {
                        if (pending >= 1) wait_vmcnt<LPC>();
                        else wait_vmcnt<0>();
                    } else {
                        (void)pending;
                        wait_vmcnt<0>();
                    }
                    __syncthreads();
                    if (c + S - 1 < nsl) {
                        issue_a(c + S - 1);
                        issue_b(c + S - 1);
                    }
                    compute(c);
                }
            }
            __syncthreads();

            if (a.ksplit > 1) {
                // split K: store this slice's raw partial tile; the reduction follows the rounds.
                // Layout: fragment (logical wave, i, jn), then quarter q of the lane's NACC
                // accumulators, then lane: each 16-byte agent-scope (device-coherent) store
                // instruction writes 1 KB contiguous; the reducing slice reads every slice back
                // in the same layout.
                const __amdgpu_buffer_rsrc_t rp =
                    __builtin_amdgcn_make_buffer_rsrc(part, (short)0, (int)(TM * TN * sizeof(float)), 0x00020000);
#pragma unroll
                for (int s = 0; s < SL; ++s) {
                    const int lam = (rd * SL + s) * P + pw;
                    trace_wave(sh, t, lam, pw, rd * SL + s);
#pragma unroll
                    for (int i = 0; i < BM; ++i)
#pragma unroll
                        for (int jn = 0; jn < BN; ++jn) {
                            const int f = (lam * BM + i) * BN + jn;
#pragma unroll
                            for (int q = 0; q < MF::NACC / 4; ++q) {
                                const f32x4 v = {acc[s][i][jn][4 * q], acc[s][i][jn][4 * q + 1], acc[s][i][jn][4 * q + 2],
                                                 acc[s][i][jn][4 * q + 3]};
                                const uint32_t fo = (uint32_t)((f * (MF::NACC / 4) + q) * kWave + lane) * 16u;
                                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(u32x4, v), rp, (int)fo, 0,
                                                                       kAgentCoherent);
                            }
                        }
                }
                continue;
            }
            epilogue(rd, acc);
        }

        if (a.ksplit > 1) {
            // count this slice's arrival; the last slice of the output tile reduces all of
            // them in slice order 0, 1, ..., ksplit-1 (same order whichever workgroup it is)
            // The partials were written with agent-scope (device-coherent) stores; waiting for
            // them to complete before the arrival is counted orders them before the count, and
            // the reducer reads them back with agent-scope loads, so no cache-wide fence is needed.
            // the arrival flag: a shared word of its own, or with split rings the first word of the
            // ring, free once the K loop has ended (the split-K path stages no epilogue there)
            int *s_lastp;
            if constexpr (SR) {
                s_lastp = reinterpret_cast<int *>(smem_);
            } else {
                __shared__ int s_last;
                s_lastp = &s_last;
            }
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
            if (tid == 0) {
                const int prev = __hip_atomic_fetch_add(a.counters + otile, 1, __ATOMIC_RELAXED,
                                                        __HIP_MEMORY_SCOPE_AGENT);
                *s_lastp = prev == a.ksplit - 1;
                if (*s_lastp) __hip_atomic_store(a.counters + otile, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            __syncthreads();
            const bool last = *s_lastp;
            // the epilogue's staging may overwrite the flag's word
            __syncthreads();
            if (last) {
                // each round's accumulators = the slices' partials added in slice order, read in
                // the fragment layout they were written in; then the regular epilogue
                const float *const base = a.work + (int64_t)otile * a.ksplit * (TM * TN);
                const __amdgpu_buffer_rsrc_t rb = __builtin_amdgcn_make_buffer_rsrc(
                    const_cast<float *>(base), (short)0, (int)((int64_t)a.ksplit * TM * TN * sizeof(float)), 0x00020000);
                for (int rd = 0; rd < ROUNDS; ++rd) {
                    acc_t acc[SL][BM][BN];
#pragma unroll
                    for (int s = 0; s < SL; ++s) {
                        const int lam = (rd * SL + s) * P + pw;
#pragma unroll
                        for (int i = 0; i < BM; ++i)
#pragma unroll
                            for (int jn = 0; jn < BN; ++jn) {
                                const int f = (lam * BM + i) * BN + jn;
#pragma unroll
                                for (int q = 0; q < MF::NACC / 4; ++q) {
                                    const uint32_t fo = (uint32_t)((f * (MF::NACC / 4) + q) * kWave + lane) * 16u;
                                    auto ld = [&](int sl) {
                                        return __builtin_bit_cast(
                                            f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                                       rb, (int)(fo + (uint32_t)sl * (TM * TN * 4u)), 0, kAgentCoherent));
                                    };
                                    f32x4 v;
                                    if (a.ksplit <= 4) {
                                        // all four loads in flight (slices past ksplit re-read
                                        // the last one and are not added)
                                        f32x4 w[4];
#pragma unroll
                                        for (int sl = 0; sl < 4; ++sl) w[sl] = ld(sl < a.ksplit ? sl : a.ksplit - 1);
                                        v = w[0];
#pragma unroll
                                        for (int sl = 1; sl < 4; ++sl) v = sl < a.ksplit ? v + w[sl] : v;
                                    } else {
                                        v = ld(0);
                                        for (int sl = 1; sl < a.ksplit; ++sl) v = v + ld(sl);
                                    }
#pragma unroll
                                    for (int e = 0; e < 4; ++e) acc[s][i][jn][4 * q + e] = v[e];
                                }
                            }
                    }
                    epilogue(rd, acc);
                }
            }
        }
    }
}

template <class T, int TM, int TN, int MS, bool UNI, bool MI = false>
inline void igemm_dma_table(const void *out[3], int *lds) {
    out[0] = reinterpret_cast<const void *>(&igemm_dma_kernel<T, TM, TN, MS, 1, UNI, MI>);
    out[1] = reinterpret_cast<const void *>(&igemm_dma_kernel<T, TM, TN, MS, 2, UNI, MI>);
    out[2] = reinterpret_cast<const void *>(&igemm_dma_kernel<T, TM, TN, MS, 4, UNI, MI>);
    *lds = DmaKernel<T, TM, TN, MS, 4>::LDS_BYTES;
}

template <class T, bool UNI>
inline int igemm_dma_table_cfg(int cfg, const void *out[3], int *lds) {
    switch (cfg) {
    case CFG_32: igemm_dma_table<T, 32, 32, 16, UNI>(out, lds); return 0;
    case CFG_64: igemm_dma_table<T, 64, 64, 32, UNI>(out, lds); return 0;
    case CFG_128: igemm_dma_table<T, 128, 128, 32, UNI>(out, lds); return 0;
    case CFG_128x64: igemm_dma_table<T, 128, 64, 32, UNI>(out, lds); return 0;
    case CFG_256x128: igemm_dma_table<T, 256, 128, 32, UNI>(out, lds); return 0;
    default: return -1;
    }
}

// Memory-based index variants (tiles 32x32, 64x64, 128x128, 128x64).
template <class T>
inline int igemm_dma_mi_table_cfg(int cfg, bool uni, const void *out[3], int *lds) {
    switch (cfg) {
    case CFG_32: uni ? igemm_dma_table<T, 32, 32, 16, true, true>(out, lds) : igemm_dma_table<T, 32, 32, 16, false, true>(out, lds); return 0;
    case CFG_64: uni ? igemm_dma_table<T, 64, 64, 32, true, true>(out, lds) : igemm_dma_table<T, 64, 64, 32, false, true>(out, lds); return 0;
    case CFG_128: uni ? igemm_dma_table<T, 128, 128, 32, true, true>(out, lds) : igemm_dma_table<T, 128, 128, 32, false, true>(out, lds); return 0;
    case CFG_128x64: uni ? igemm_dma_table<T, 128, 64, 32, true, true>(out, lds) : igemm_dma_table<T, 128, 64, 32, false, true>(out, lds); return 0;
    default: return -1;
    }
}

}  // namespace miriam
