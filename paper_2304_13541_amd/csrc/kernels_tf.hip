// Transformer kernels of the BERT encoder (Sec. 4.4's transformer workload):
// token embedding + layer norm, layer norm, and the multi-head
// self-attention core.  The encoder's matrix products run on the
// implicit-GEMM convolution kernel as 1x1 convolutions (bias, residual,
// GELU and tanh in its epilogue).
//
// Layer norm (both kernels): one 256-thread block per token row; the row's
// values stay in registers, mean and (biased) variance are fp32 block
// reductions (wave shuffles, then one LDS value per wave), output bf16.
//
// Attention: one block per (head, sequence).  Queries, keys and values of
// the sequence's T <= 48 tokens (64 dims per head) are read from the fused
// q|k|v projection [tokens][3 * width] into LDS as fp32; the T x T scores
// q_i . k_j / 8 are formed in LDS, each row is turned into softmax weights
// by one wave (max, exp, sum), and the outputs o_i = sum_j p_ij v_j are
// written as bf16 at the head's columns of [tokens][width].  The sequence is
// short (tens of tokens), so this is plain fp32 vector arithmetic.
#include "common.hpp"

namespace dstack {

namespace {

constexpr int LN_MAX_PER_THREAD = 8;  // rows of up to 2048 values
constexpr int ATT_DH = 64;            // head width
constexpr int ATT_MAX_T = 48;         // tokens per sequence (the four arrays fit 64 KB of LDS)

__device__ __forceinline__ float wave_sum(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v += __shfl_xor(v, o, 64);
  return v;
}
__device__ __forceinline__ float wave_max(float v) {
#pragma unroll
  for (int o = 32; o >= 1; o >>= 1) v = fmaxf(v, __shfl_xor(v, o, 64));
  return v;
}

// sum over the 256-thread block (every thread gets the total)
__device__ __forceinline__ float block_sum(float v, float* red) {
  v = wave_sum(v);
  const int wave = threadIdx.x >> 6;
  __syncthreads();  // red may still be read from the previous call
  if ((threadIdx.x & 63) == 0) red[wave] = v;
  __syncthreads();
  return red[0] + red[1] + red[2] + red[3];
}

// normalise the thread's values of one row of H and write them as bf16
__device__ __forceinline__ void ln_row(float (&v)[LN_MAX_PER_THREAD], int H, const float* gamma, const float* beta,
                                       float eps, bf16* y, float* red) {
  float s = 0.f;
#pragma unroll
  for (int j = 0; j < LN_MAX_PER_THREAD; ++j)
    if ((int)threadIdx.x + j * 256 < H) s += v[j];
  const float mean = block_sum(s, red) / (float)H;
  float q = 0.f;
#pragma unroll
  for (int j = 0; j < LN_MAX_PER_THREAD; ++j)
    if ((int)threadIdx.x + j * 256 < H) q += (v[j] - mean) * (v[j] - mean);
  const float inv = rsqrtf(block_sum(q, red) / (float)H + eps);
#pragma unroll
  for (int j = 0; j < LN_MAX_PER_THREAD; ++j) {
    const int c = threadIdx.x + j * 256;
    if (c < H) {
      float o = (v[j] - mean) * inv;
      if (gamma) o *= gamma[c];
      if (beta) o += beta[c];
      y[c] = (bf16)o;
    }
  }
}

__global__ __launch_bounds__(256) void embed_ln_kernel(const int* __restrict__ ids, int T, int vocab,
                                                       const bf16* __restrict__ we, const bf16* __restrict__ pe,
                                                       const bf16* __restrict__ te, int H, const float* gamma,
                                                       const float* beta, float eps, bf16* __restrict__ y) {
  __shared__ float red[4];
  const int row = blockIdx.x;
  const int t = row % T;
  const int id = min(max(ids[row], 0), vocab - 1);  // ids outside the vocabulary read its last row
  float v[LN_MAX_PER_THREAD];
#pragma unroll
  for (int j = 0; j < LN_MAX_PER_THREAD; ++j) {
    const int c = threadIdx.x + j * 256;
    v[j] = c < H ? (float)we[(long)id * H + c] + (float)pe[(long)t * H + c] + (float)te[c] : 0.f;
  }
  ln_row(v, H, gamma, beta, eps, y + (long)row * H, red);
}

__global__ __launch_bounds__(256) void layernorm_kernel(const bf16* __restrict__ x, int H, const float* gamma,
                                                        const float* beta, float eps, bf16* __restrict__ y) {
  __shared__ float red[4];
  const long row = blockIdx.x;
  float v[LN_MAX_PER_THREAD];
#pragma unroll
  for (int j = 0; j < LN_MAX_PER_THREAD; ++j) {
    const int c = threadIdx.x + j * 256;
    v[j] = c < H ? (float)x[row * H + c] : 0.f;
  }
  ln_row(v, H, gamma, beta, eps, y + row * H, red);
}

__global__ __launch_bounds__(256) void attention_kernel(const bf16* __restrict__ qkv, int T, int width,
                                                        bf16* __restrict__ out) {
  __shared__ float q[ATT_MAX_T][ATT_DH + 1], k[ATT_MAX_T][ATT_DH + 1], v[ATT_MAX_T][ATT_DH + 1];
  __shared__ float p[ATT_MAX_T][ATT_MAX_T + 1];
  const int h = blockIdx.x, b = blockIdx.y, tid = threadIdx.x;
  const long tok0 = (long)b * T;
  for (int i = tid; i < T * ATT_DH; i += 256) {
    const int r = i / ATT_DH, e = i - r * ATT_DH;
    const bf16* src = qkv + (tok0 + r) * 3 * width + h * ATT_DH + e;
    q[r][e] = (float)src[0];
    k[r][e] = (float)src[width];
    v[r][e] = (float)src[2 * width];
  }
  __syncthreads();
  const float scale = 0.125f;  // 1 / sqrt(64)
  for (int i = tid; i < T * T; i += 256) {
    const int r = i / T, c = i - r * T;
    float d = 0.f;
#pragma unroll 16
    for (int e = 0; e < ATT_DH; ++e) d += q[r][e] * k[c][e];
    p[r][c] = d * scale;
  }
  __syncthreads();
  const int lane = tid & 63, wave = tid >> 6;
  for (int r = wave; r < T; r += 4) {  // one wave per row: lane j holds key j
    const float s = lane < T ? p[r][lane] : -INFINITY;
    const float mx = wave_max(s);
    const float ex = lane < T ? __expf(s - mx) : 0.f;
    const float sum = wave_sum(ex);
    if (lane < T) p[r][lane] = ex / sum;
  }
  __syncthreads();
  for (int i = tid; i < T * ATT_DH; i += 256) {
    const int r = i / ATT_DH, e = i - r * ATT_DH;
    float o = 0.f;
    for (int j = 0; j < T; ++j) o += p[r][j] * v[j][e];
    out[(tok0 + r) * width + h * ATT_DH + e] = (bf16)o;
  }
}

}  // namespace

dstack_status launch_embed_ln(const int* ids, int rows, int T, int vocab, const bf16* we, const bf16* pe,
                              const bf16* te, int H, const float* gamma, const float* beta, float eps, bf16* y,
                              hipStream_t st) {
  DS_CHECK(ids && we && pe && te && y, DSTACK_E_INVALID, "embed_ln: null pointer");
  DS_CHECK(rows > 0 && T > 0 && vocab > 0 && H > 0, DSTACK_E_INVALID, "embed_ln: bad shape");
  DS_CHECK(H <= 256 * LN_MAX_PER_THREAD, DSTACK_E_UNSUPPORTED, "embed_ln: width above 2048");
  launch(embed_ln_kernel, dim3((unsigned)rows), dim3(256), 0, st, ids, T, vocab, we, pe, te, H, gamma, beta, eps, y);
  DS_HIP(hipGetLastError());
  return DSTACK_OK;
}

dstack_status launch_layernorm(const bf16* x, int rows, int H, const float* gamma, const float* beta, float eps,
                               bf16* y, hipStream_t st) {
  DS_CHECK(x && y, DSTACK_E_INVALID, "layernorm: null pointer");
  DS_CHECK(rows > 0 && H > 0, DSTACK_E_INVALID, "layernorm: bad shape");
  DS_CHECK(H <= 256 * LN_MAX_PER_THREAD, DSTACK_E_UNSUPPORTED, "layernorm: width above 2048");
  launch(layernorm_kernel, dim3((unsigned)rows), dim3(256), 0, st, x, H, gamma, beta, eps, y);
  DS_HIP(hipGetLastError());
  return DSTACK_OK;
}

dstack_status launch_attention(const bf16* qkv, int B, int T, int heads, int dh, bf16* out, hipStream_t st) {
  DS_CHECK(qkv && out, DSTACK_E_INVALID, "attention: null pointer");
  DS_CHECK(B > 0 && T > 0 && heads > 0, DSTACK_E_INVALID, "attention: bad shape");
  DS_CHECK(dh == ATT_DH && T <= ATT_MAX_T && heads <= 65535 && B <= 65535, DSTACK_E_UNSUPPORTED,
           "attention: head width 64 and at most 48 tokens");
  launch(attention_kernel, dim3((unsigned)heads, (unsigned)B), dim3(256), 0, st, qkv, T, heads * dh, out);
  DS_HIP(hipGetLastError());
  return DSTACK_OK;
}

}  // namespace dstack
