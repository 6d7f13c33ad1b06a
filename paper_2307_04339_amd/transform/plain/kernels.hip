// Plain (non-elastic) HIP kernels of the kind the source-to-source transformer takes as
// input: 1-D grids, one logical block per blockIdx.x, written without any knowledge of
// shards.  Each is preceded by a line "// elastic: block N" naming the block size it is
// written for (its logical block).  The transformer derives the elastic forms from this file.

// y = max(x + b[c], 0) over an N x C row-major matrix, one element per thread.
// elastic: block 256
__global__ void plain_bias_relu(const float *x, const float *b, float *y, int n, int c) {
    const int i = blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= n) return;
    const float v = x[i] + b[i % c];
    y[i] = v > 0.0f ? v : 0.0f;
}

// 2x2 / stride-2 max pooling of an NHWC image, one output element per thread, written as a
// grid-stride loop over the whole output (so it also reads gridDim.x).
// elastic: block 128
__global__ void plain_maxpool2(const float *x, float *y, int n, int h, int w, int c) {
    const int ho = h / 2, wo = w / 2;
    const int total = n * ho * wo * c;
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < total; i += gridDim.x * blockDim.x) {
        const int ch = i % c, q = (i / c) % wo, p = (i / (c * wo)) % ho, img = i / (c * wo * ho);
        const float *src = x + (((long long)img * h + 2 * p) * w + 2 * q) * c + ch;
        const float a = fmaxf(src[0], src[c]);
        const float d = fmaxf(src[(long long)w * c], src[(long long)w * c + c]);
        y[i] = fmaxf(a, d);
    }
}

// C = A B (M x K times K x N, row-major) with 16 x 16 output tiles through shared memory;
// tile t of the flattened grid covers tile row t / ceil(N / 16) and tile column t % ceil(N / 16).
// It synchronises its block, so its elastic form keeps the 256-thread block.
// elastic: block 256
__global__ void plain_tiled_gemm(const float *A, const float *B, float *C, int M, int N, int K) {
    __shared__ float As[16][17];
    __shared__ float Bs[16][17];
    const int nT = (N + 15) / 16;
    const int bm = blockIdx.x / nT, bn = blockIdx.x % nT;
    const int ty = threadIdx.x / 16, tx = threadIdx.x % 16;
    const int row = bm * 16 + ty, col = bn * 16 + tx;
    float acc = 0.0f;
    for (int k0 = 0; k0 < K; k0 += 16) {
        As[ty][tx] = (row < M && k0 + tx < K) ? A[(long long)row * K + k0 + tx] : 0.0f;
        Bs[ty][tx] = (k0 + ty < K && col < N) ? B[(long long)(k0 + ty) * N + col] : 0.0f;
        __syncthreads();
        for (int kk = 0; kk < 16; ++kk) acc += As[ty][kk] * Bs[kk][tx];
        __syncthreads();
    }
    if (row < M && col < N) C[(long long)row * N + col] = acc;
}

// y = a * x + (x one column to the right, zero past the edge) over an R x C row-major image,
// one element per thread on a 2-D grid of 32 x 8 blocks.
// elastic: block 32x8
__global__ void plain_shift_add2d(const float *x, float *y, int rows, int cols, float a) {
    const int c = blockIdx.x * blockDim.x + threadIdx.x;
    const int r = blockIdx.y * blockDim.y + threadIdx.y;
    if (r >= rows || c >= cols) return;
    const float right = c + 1 < cols ? x[(long long)r * cols + c + 1] : 0.0f;
    y[(long long)r * cols + c] = a * x[(long long)r * cols + c] + right;
}

// out = in transposed (R x C -> C x R) through a 16 x 17 shared tile on a 2-D grid of 16 x 16
// blocks; it synchronises its block, so its elastic form keeps the 256-thread block.
// elastic: block 16x16
__global__ void plain_transpose16(const float *in, float *out, int rows, int cols) {
    __shared__ float tile[16][17];
    const int c = blockIdx.x * 16 + threadIdx.x, r = blockIdx.y * 16 + threadIdx.y;
    if (r < rows && c < cols) tile[threadIdx.y][threadIdx.x] = in[(long long)r * cols + c];
    __syncthreads();
    const int oc = blockIdx.y * 16 + threadIdx.x, orow = blockIdx.x * 16 + threadIdx.y;
    if (orow < cols && oc < rows) out[(long long)orow * rows + oc] = tile[threadIdx.x][threadIdx.y];
}
