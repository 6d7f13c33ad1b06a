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

// Direct 3x3 convolution, NHWC input [n, h, w, c], weights [k, 3, 3, c], zero padding 1, stride
// s, plus bias and ReLU; one output element per thread, taps row-major and channels innermost.
// elastic: block 256
__global__ void plain_conv3x3_relu(const float *x, const float *wt, const float *b, float *y, int n, int h, int w,
                                   int c, int k, int s) {
    const int ho = (h + 2 - 3) / s + 1, wo = (w + 2 - 3) / s + 1;
    const long long total = (long long)n * ho * wo * k;
    const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= total) return;
    const int oc = (int)(i % k), q = (int)((i / k) % wo), p = (int)((i / ((long long)k * wo)) % ho);
    const int img = (int)(i / ((long long)k * wo * ho));
    float acc = 0.0f;
    for (int r = 0; r < 3; ++r) {
        const int hi = p * s - 1 + r;
        if (hi < 0 || hi >= h) continue;
        for (int t = 0; t < 3; ++t) {
            const int wi = q * s - 1 + t;
            if (wi < 0 || wi >= w) continue;
            const float *xp = x + (((long long)img * h + hi) * w + wi) * c;
            const float *wp = wt + ((long long)(oc * 3 + r) * 3 + t) * c;
            for (int ch = 0; ch < c; ++ch) acc = fmaf(xp[ch], wp[ch], acc);
        }
    }
    const float v = acc + b[oc];
    y[i] = v > 0.0f ? v : 0.0f;
}

// Depthwise 3x3 convolution (MobileNet), NHWC [n, h, w, c], weights [c, 3, 3], zero padding 1,
// stride s, plus bias and ReLU6; one output element per thread.
// elastic: block 256
__global__ void plain_dwconv3x3_relu6(const float *x, const float *wt, const float *b, float *y, int n, int h, int w,
                                      int c, int s) {
    const int ho = (h + 2 - 3) / s + 1, wo = (w + 2 - 3) / s + 1;
    const long long total = (long long)n * ho * wo * c;
    const long long i = (long long)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= total) return;
    const int ch = (int)(i % c), q = (int)((i / c) % wo), p = (int)((i / ((long long)c * wo)) % ho);
    const int img = (int)(i / ((long long)c * wo * ho));
    float acc = 0.0f;
    for (int r = 0; r < 3; ++r) {
        const int hi = p * s - 1 + r;
        if (hi < 0 || hi >= h) continue;
        for (int t = 0; t < 3; ++t) {
            const int wi = q * s - 1 + t;
            if (wi < 0 || wi >= w) continue;
            acc = fmaf(x[(((long long)img * h + hi) * w + wi) * c + ch], wt[(ch * 3 + r) * 3 + t], acc);
        }
    }
    const float v = acc + b[ch];
    y[i] = fminf(fmaxf(v, 0.0f), 6.0f);
}

// Softmax of each row of a rows x n matrix (attention scores), one 256-thread block per row:
// the row maximum and the sum of exponentials are reduced in shared memory, so the elastic
// form keeps the 256-thread block.
// elastic: block 256
__global__ void plain_softmax_rows(const float *x, float *y, int rows, int n) {
    __shared__ float red[256];
    const int row = blockIdx.x;
    if (row >= rows) return;
    const float *xr = x + (long long)row * n;
    float m = -INFINITY;
    for (int j = threadIdx.x; j < n; j += 256) m = fmaxf(m, xr[j]);
    red[threadIdx.x] = m;
    __syncthreads();
    for (int d = 128; d > 0; d >>= 1) {
        if (threadIdx.x < d) red[threadIdx.x] = fmaxf(red[threadIdx.x], red[threadIdx.x + d]);
        __syncthreads();
    }
    m = red[0];
    __syncthreads();
    float sum = 0.0f;
    for (int j = threadIdx.x; j < n; j += 256) sum += expf(xr[j] - m);
    red[threadIdx.x] = sum;
    __syncthreads();
    for (int d = 128; d > 0; d >>= 1) {
        if (threadIdx.x < d) red[threadIdx.x] += red[threadIdx.x + d];
        __syncthreads();
    }
    const float inv = 1.0f / red[0];
    for (int j = threadIdx.x; j < n; j += 256) y[(long long)row * n + j] = expf(xr[j] - m) * inv;
}

// LayerNorm of each row of a rows x n matrix (transformer), one 128-thread block per row: mean
// and variance reduced in shared memory, then y = (x - mean) / sqrt(var + eps) * g + b.
// elastic: block 128
__global__ void plain_layernorm_rows(const float *x, const float *g, const float *b, float *y, int rows, int n,
                                     float eps) {
    __shared__ float red[128];
    const int row = blockIdx.x;
    if (row >= rows) return;
    const float *xr = x + (long long)row * n;
    float s = 0.0f;
    for (int j = threadIdx.x; j < n; j += 128) s += xr[j];
    red[threadIdx.x] = s;
    __syncthreads();
    for (int d = 64; d > 0; d >>= 1) {
        if (threadIdx.x < d) red[threadIdx.x] += red[threadIdx.x + d];
        __syncthreads();
    }
    const float mean = red[0] / (float)n;
    __syncthreads();
    float v = 0.0f;
    for (int j = threadIdx.x; j < n; j += 128) {
        const float d = xr[j] - mean;
        v += d * d;
    }
    red[threadIdx.x] = v;
    __syncthreads();
    for (int d = 64; d > 0; d >>= 1) {
        if (threadIdx.x < d) red[threadIdx.x] += red[threadIdx.x + d];
        __syncthreads();
    }
    const float rstd = 1.0f / sqrtf(red[0] / (float)n + eps);
    for (int j = threadIdx.x; j < n; j += 128) y[(long long)row * n + j] = (xr[j] - mean) * rstd * g[j] + b[j];
}
