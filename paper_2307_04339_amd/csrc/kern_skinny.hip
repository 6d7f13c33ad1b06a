// Elastic kernel for skinny products (fully connected layers at small batch):
// Y[m][n] = sum_k X[m][k] * W[n][k] with M <= 16.  Such a product is bound by
// streaming W from HBM, so the logical tile is 16 output columns (all M rows)
// and the K range is split into 4 fixed quarters, one per logical wave; each
// wave streams its quarter of the 16 weight rows with 16-byte loads straight
// into MFMA 16x16x32 operands (no LDS staging: nothing is reused), and the 4
// partial sums are added in fixed order (wave 0 + 1 + 2 + 3) through LDS before
// the epilogue.  The split and the order depend only on K, never on the shard,
// grid or physical block, so results stay bit-identical across elastic
// configurations.
//
// Split K (ksplit > 1): tile id = output tile * ksplit + slice, slice s covering
// [s L, (s+1) L) of K with L a whole number of wave groups.  Each slice writes its
// 16 x 16 partial (the fixed-order sum of its quarters) with device-coherent stores;
// the last slice to arrive at the output tile (relaxed device-scope counter) adds the
// partials in slice order 0, 1, ..., ksplit-1, applies the epilogue and resets the
// counter.  The order does not depend on which workgroup arrives last, so results stay
// bit-identical across elastic configurations; every pass over the op must cover its
// whole tile space.  More, shorter tiles let a small-batch FC layer fill the GPU and be
// sharded without serialising weight streams.
//
// K-order inside a wave: MFMA step j of a group covers the 32 consecutive elements
// [k0 + 32 j, k0 + 32 j + 32), k-group g of the lanes holding [k0 + 32 j + 8 g, +8),
// so one load instruction reads 64 contiguous bytes of each of the 16 weight rows.
// The next group's loads are issued before the current group's MFMAs, so two groups
// (8 KB of weights per wave) are in flight.
#include "elastic_common.h"
#include "igemm.h"

namespace miriam {

constexpr int kSkinnyTN = 16;

template <class T, int P>
__global__ __launch_bounds__(kWave * P) void skinny_kernel(IgemmArgs a, Shard sh) {
    typedef Mfma<T, 16> MF;
    typedef typename MF::op_t op_t;
    constexpr int NJ = 4;              // MFMA steps per group
    constexpr int GROUP = 32 * NJ;     // K consumed by one group
    __shared__ float part[kLogicalWaves][16][17];

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
    TileDigits<2> td;
    {
        const uint32_t radix[2] = {(uint32_t)ks, 0u};
        td.init((uint32_t)(sh.begin + rank), (uint32_t)G, radix);
    }

    int iter = 0;
    for (int64_t t = sh.begin + rank; t < sh.begin + sh.len; t += G, ++iter, td.advance()) {
        trace_tile(sh, t, iter);
        const int slice = (int)td.d[0];
        const int64_t otile = td.d[1];
        const int64_t n0 = otile * kSkinnyTN;
        const int64_t sb = slice * ls, se = sb + ls < a.K ? sb + ls : a.K;
        const int64_t n = n0 + row;
        const bool a_ok = row < a.M, b_ok = n < a.Nc;
        const T *xr = X + (int64_t)row * a.ldx;
        const T *wr = Wt + n * a.ldw;
        for (int s = 0; s < kLogicalWaves / P; ++s) {
            const int lam = s * P + pw;
            trace_wave(sh, t, lam, pw, s);
            const int64_t kb = sb + lam * kq;
            const int64_t ke = kb + kq < se ? kb + kq : se;
            f32x4 acc = {0.0f, 0.0f, 0.0f, 0.0f};
            Vec16<T> av[NJ], bv[NJ], an[NJ], bn_[NJ];
            auto load = [&](int64_t k0, Vec16<T> *ao, Vec16<T> *bo) {
#pragma unroll
                for (int j = 0; j < NJ; ++j) {
                    const int64_t k = k0 + j * 32 + grp * 8;
                    const bool kin = k + 8 <= ke;
                    ao[j] = (a_ok && kin) ? ld_vec(xr + k) : zero_vec<T>();
                    bo[j] = (b_ok && kin) ? ld_vec(wr + k) : zero_vec<T>();
                }
            };
            int64_t k0 = kb;
            if (k0 < ke) load(k0, av, bv);
            while (k0 < ke) {
                const int64_t k1 = k0 + GROUP;
                if (k1 < ke) load(k1, an, bn_);
#pragma unroll
                for (int j = 0; j < NJ; ++j)
                    acc = MF::run(*reinterpret_cast<const op_t *>(&av[j].u), *reinterpret_cast<const op_t *>(&bv[j].u), acc);
#pragma unroll
                for (int j = 0; j < NJ; ++j) {
                    av[j] = an[j];
                    bv[j] = bn_[j];
                }
                k0 = k1;
            }
            // 16x16 accumulator: lane holds column (lane % 16), rows 4 * (lane / 16) + e
#pragma unroll
            for (int e = 0; e < 4; ++e) part[lam][4 * grp + e][row] = acc[e];
        }
        __syncthreads();
        if (ks > 1) {
            // partial of this slice -> workspace; the last slice of the output tile reduces
            float *const wp = a.work + (otile * ks + slice) * (16 * kSkinnyTN);
            for (int idx = tid; idx < 16 * kSkinnyTN; idx += kWave * P) {
                const int m = idx / kSkinnyTN, c = idx % kSkinnyTN;
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
                const float *const wb = a.work + otile * ks * (16 * kSkinnyTN);
                for (int idx = tid; idx < 16 * kSkinnyTN; idx += kWave * P) {
                    const int m = idx / kSkinnyTN, c = idx % kSkinnyTN;
                    const int64_t nn = n0 + c;
                    if (m < a.M && nn < a.Nc) {
                        float v = __hip_atomic_load(wb + idx, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        for (int q = 1; q < ks; ++q)
                            v += __hip_atomic_load(wb + q * (16 * kSkinnyTN) + idx, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
                        const int64_t off = m * a.ldy + nn;
                        const float res = (a.epi.flags & EPI_RES) ? ld_f(R + off) : 0.0f;
                        st_f(Y + off, epilogue_apply(a.epi, v, nn, res));
                    }
                }
            }
        } else {
            for (int idx = tid; idx < 16 * kSkinnyTN; idx += kWave * P) {
                const int m = idx / kSkinnyTN, c = idx % kSkinnyTN;
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

template <class T>
static void skinny_table(const void *out[3]) {
    out[0] = reinterpret_cast<const void *>(&skinny_kernel<T, 1>);
    out[1] = reinterpret_cast<const void *>(&skinny_kernel<T, 2>);
    out[2] = reinterpret_cast<const void *>(&skinny_kernel<T, 4>);
}

int skinny_kernels(int dtype, const void *out[3]) {
    switch (dtype) {
    case 1: skinny_table<half_t>(out); return 0;
    case 2: skinny_table<bf16_t>(out); return 0;
    default: return -1;
    }
}

}  // namespace miriam
