// Elastic kernel for skinny products (fully connected layers at small batch):
// Y[m][n] = sum_k X[m][k] * W[n][k] with M <= 16.  Such a product is bound by
// streaming W from HBM.  The logical tile is CG groups of 16 output columns (all M
// rows), and the K range is split into 4 fixed quarters, one per logical wave; each
// wave streams its quarter of the tile's 16 CG weight rows with 16-byte loads straight
// into MFMA 16x16x32 operands (no LDS staging: nothing is reused), one load of the
// activations feeding the CG column groups, and the 4 partial sums are added in fixed
// order (wave 0 + 1 + 2 + 3) through LDS before the epilogue.  Wider tiles (CG > 1)
// cut the activation loads, which every column tile repeats over its K range, to one
// per CG weight loads.  The split and the order depend only on K, never on the shard,
// grid or physical block, so results stay bit-identical across elastic
// configurations.
//
// Split K (ksplit > 1): tile id = output tile * ksplit + slice, slice s covering
// [s L, (s+1) L) of K with L a whole number of wave groups.  Each slice writes its
// 16 x 16 CG partial (the fixed-order sum of its quarters) with device-coherent stores;
// the last slice to arrive at the output tile (relaxed device-scope counter) adds the
// partials in slice order 0, 1, ..., ksplit-1, applies the epilogue and resets the
// counter.  The order does not depend on which workgroup arrives last, so results stay
// bit-identical across elastic configurations; every pass over the op must cover its
// whole tile space.  More, shorter tiles let a small-batch FC layer fill the GPU and be
// sharded without serialising weight streams.
//
// K-order inside a wave: MFMA step j of a group covers the 32 consecutive elements
// [k0 + 32 j, k0 + 32 j + 32), k-group g of the lanes holding [k0 + 32 j + 8 g, +8),
// so one load instruction reads 64 contiguous bytes of each of 16 rows.  A group is
// NJ steps; a wave takes the groups of its quarter in a rotation fixed by the tile id,
// and the next group's loads are issued before the current group's MFMAs, so two
// groups are in flight.
#include "elastic_common.h"
#include "igemm.h"

namespace miriam {

template <class T, int P, int CG, int NJ>
__global__ __launch_bounds__(kWave * P, 4) void skinny_kernel(IgemmArgs a, Shard sh) {
    typedef Mfma<T, 16> MF;
    typedef typename MF::op_t op_t;
    constexpr int GROUP = 32 * NJ;       // K consumed by one group
    constexpr int TN = 16 * CG;          // output columns per tile
    constexpr uint32_t ES = sizeof(T);
    constexpr uint32_t OOR = 0x80000000u;  // past both operand windows: the load returns zeros
    __shared__ float part[kLogicalWaves][16][TN + 1];

    const int tid = threadIdx.x;
    const int pw = __builtin_amdgcn_readfirstlane(tid / kWave);
    const int lane = tid % kWave;
    const T *__restrict__ X = static_cast<const T *>(a.x);
    const T *__restrict__ Wt = static_cast<const T *>(a.w);
    T *__restrict__ Y = static_cast<T *>(a.y);
    const T *__restrict__ R = static_cast<const T *>(a.res);
    __shared__ int s_last;
    const int ks = a.ksplit;
    // slice length and quarter length, whole numbers of groups
    const int64_t ls = ((a.K + (int64_t)ks * 4 * GROUP - 1) / ((int64_t)ks * 4 * GROUP)) * 4 * GROUP;
    const int64_t kq = ls / 4;
    const int64_t G = gridDim.x;
    const int64_t rank = wg_rank(blockIdx.x, G);
    const int row = lane % 16, grp = lane / 16;
    // Operands are read as buffers with 32-bit byte offsets (the library admits the kernel only
    // when the activations and a tile's weight rows span less than 2^31 bytes): the lane's row
    // and k-group fixed in the vector offset, the group's K start in the scalar offset.  Rows
    // past M or N and K past the wave's range take an offset outside the window, which reads
    // zeros, so the loads need no branches.
    const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(const_cast<T *>(X), (short)0, 0x7FFFFFFF, 0x00020000);
    const uint32_t vx = row < a.M ? (uint32_t)(((int64_t)row * a.ldx + grp * 8) * ES) : OOR;
    const int kl = grp * 8 + 8;  // end of the lane's 8 K values within an MFMA step
    TileDigits<2> td;
    {
        const uint32_t radix[2] = {(uint32_t)ks, 0u};
        td.init((uint32_t)(sh.begin + rank), (uint32_t)G, radix);
    }

    struct Grp {
        u32x4 x[NJ];
        u32x4 w[CG][NJ];
    };
    int iter = 0;
    for (int64_t t = sh.begin + rank; t < sh.begin + sh.len; t += G, ++iter, td.advance()) {
        trace_tile(sh, t, iter);
        const int slice = (int)td.d[0];
        const int64_t otile = td.d[1];
        const int64_t n0 = otile * TN;
        const int64_t sb = slice * ls, se = sb + ls < a.K ? sb + ls : a.K;
        const __amdgpu_buffer_rsrc_t rw =
            __builtin_amdgcn_make_buffer_rsrc(const_cast<T *>(Wt + n0 * a.ldw), (short)0, 0x7FFFFFFF, 0x00020000);
        uint32_t vw[CG];
#pragma unroll
        for (int c = 0; c < CG; ++c)
            vw[c] = n0 + 16 * c + row < a.Nc ? (uint32_t)(((int64_t)(16 * c + row) * a.ldw + grp * 8) * ES) : OOR;
        for (int s = 0; s < kLogicalWaves / P; ++s) {
            const int lam = s * P + pw;
            trace_wave(sh, t, lam, pw, s);
            const int64_t kb = sb + lam * kq;
            const int64_t ke = kb + kq < se ? kb + kq : se;
            f32x4 acc[CG];
#pragma unroll
            for (int c = 0; c < CG; ++c) acc[c] = f32x4{0.0f, 0.0f, 0.0f, 0.0f};
            // group starting at K = k0; steps past ke read zeros
            auto issue = [&](int64_t k0, Grp &r) {
                const int64_t rem = ke - k0;
                const int so = (int)(k0 * ES);
#pragma unroll
                for (int j = 0; j < NJ; ++j) {
                    const bool kin = kl + 32 * j <= rem;
                    r.x[j] = __builtin_amdgcn_raw_buffer_load_b128(rx, (int)(kin ? vx + 32 * j * ES : OOR), so, 0);
#pragma unroll
                    for (int c = 0; c < CG; ++c)
                        r.w[c][j] = __builtin_amdgcn_raw_buffer_load_b128(rw, (int)(kin ? vw[c] + 32 * j * ES : OOR), so, 0);
                }
            };
            auto mma = [&](const Grp &r) {
#pragma unroll
                for (int j = 0; j < NJ; ++j)
#pragma unroll
                    for (int c = 0; c < CG; ++c)
                        acc[c] = MF::run(__builtin_bit_cast(op_t, r.x[j]), __builtin_bit_cast(op_t, r.w[c][j]), acc[c]);
            };
            // Groups in rotated order, starting at group (output tile mod groups): the column
            // tiles that run at the same time then read different activation lines instead of
            // all reading the same ones (VGG-16 fc6: 54.9 -> 51.1 us).  The order depends on the
            // tile id only.  Two register sets in turn, the next group's loads issued before
            // this group's MFMAs, with no branch between a group's loads and their use.
            const int ng = kb < ke ? (int)((ke - kb + GROUP - 1) / GROUP) : 0;
            const int rot = ng > 0 ? (int)(otile % ng) : 0;
            auto gk = [&](int g) {
                const int q = g + rot < ng ? g + rot : g + rot - ng;
                return kb + (int64_t)q * GROUP;
            };
            if (ng > 0) {
                Grp ra, rb;
                issue(gk(0), ra);
                int g = 0;
                for (; g + 2 < ng; g += 2) {
                    issue(gk(g + 1), rb);
                    mma(ra);
                    issue(gk(g + 2), ra);
                    mma(rb);
                }
                if (g + 1 < ng) {
                    issue(gk(g + 1), rb);
                    mma(ra);
                    mma(rb);
                } else {
                    mma(ra);
                }
            }
            // 16x16 accumulator c: lane holds column 16 c + (lane % 16), rows 4 * (lane / 16) + e
#pragma unroll
            for (int c = 0; c < CG; ++c)
#pragma unroll
                for (int e = 0; e < 4; ++e) part[lam][4 * grp + e][16 * c + row] = acc[c][e];
        }
        __syncthreads();
        if (ks > 1) {
            // partial of this slice -> workspace; the last slice of the output tile reduces
            float *const wp = a.work + (otile * ks + slice) * (16 * TN);
            for (int idx = tid; idx < 16 * TN; idx += kWave * P) {
                const int m = idx / TN, c = idx % TN;
                const float v = ((part[0][m][c] + part[1][m][c]) + part[2][m][c]) + part[3][m][c];
                __hip_atomic_store(wp + idx, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            // the partial's stores complete before the arrival is counted
            __builtin_amdgcn_s_waitcnt(0);
            __syncthreads();
            if (tid == 0) {
                const int prev = __hip_atomic_fetch_add(a.counters + otile, 1, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                s_last = prev == ks - 1;
                if (s_last) __hip_atomic_store(a.counters + otile, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
            }
            __syncthreads();
            if (s_last) {
                const float *const wb = a.work + otile * ks * (16 * TN);
                for (int idx = tid; idx < 16 * TN; idx += kWave * P) {
                    const int m = idx / TN, c = idx % TN;
                    const int64_t nn = n0 + c;
                    if (m < a.M && nn < a.Nc) {
                        float v = __hip_atomic_load(wb + idx, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        for (int q = 1; q < ks; ++q)
                            v += __hip_atomic_load(wb + q * (16 * TN) + idx, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        const int64_t off = m * a.ldy + nn;
                        const float res = (a.epi.flags & EPI_RES) ? ld_f(R + off) : 0.0f;
                        st_f(Y + off, epilogue_apply(a.epi, v, nn, res));
                    }
                }
            }
        } else {
            for (int idx = tid; idx < 16 * TN; idx += kWave * P) {
                const int m = idx / TN, c = idx % TN;
                const int64_t nn = n0 + c;
                if (m < a.M && nn < a.Nc) {
                    const float v = ((part[0][m][c] + part[1][m][c]) + part[2][m][c]) + part[3][m][c];
                    const int64_t off = m * a.ldy + nn;
                    const float res = (a.epi.flags & EPI_RES) ? ld_f(R + off) : 0.0f;
                    st_f(Y + off, epilogue_apply(a.epi, v, nn, res));
                }
            }
        }
        __syncthreads();
    }
}

template <class T, int CG, int NJ>
static void skinny_table(const void *out[3]) {
    out[0] = reinterpret_cast<const void *>(&skinny_kernel<T, 1, CG, NJ>);
    out[1] = reinterpret_cast<const void *>(&skinny_kernel<T, 2, CG, NJ>);
    out[2] = reinterpret_cast<const void *>(&skinny_kernel<T, 4, CG, NJ>);
}

template <class T>
static int skinny_table_cg(int cg, const void *out[3]) {
    switch (cg) {
    case 1: skinny_table<T, 1, 4>(out); return 0;
    case 2: skinny_table<T, 2, 2>(out); return 0;
    default: return -1;
    }
}

int skinny_kernels(int dtype, int cg, const void *out[3]) {
    switch (dtype) {
    case 1: return skinny_table_cg<half_t>(cg, out);
    case 2: return skinny_table_cg<bf16_t>(cg, out);
    default: return -1;
    }
}

int skinny_group(int cg) { return cg == 1 ? 128 : 64; }

}  // namespace miriam
