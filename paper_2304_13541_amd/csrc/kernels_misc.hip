// Memory-bound kernels of the hot path: depthwise 3x3 convolution and
// pooling.  In the paper's terms (Sec. 4.1) these are the low
// arithmetic-intensity kernels: they are written for coalesced 16-byte
// accesses along the channel (NHWC) axis, not for matrix cores.

#include "common.hpp"

namespace dstack {

__device__ __forceinline__ bf16x8 ld8(const bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }
__device__ __forceinline__ void st8(bf16* p, bf16x8 v) { *reinterpret_cast<bf16x8*>(p) = v; }

// ------------------------------------------------------------ depthwise ----
// Thread = 8 channels (one 16-byte vector) x V consecutive output pixels of
// one output row.  The 9 weight vectors stay in registers; the input rows are
// walked once each: row r contributes input columns wo0*STRIDE-1 ..
// (wo0+V-1)*STRIDE+1, every column loaded once and used by the (up to 3)
// outputs whose window covers it.  Loads per V outputs: 3 * ((V-1)*STRIDE+3)
// vectors instead of 9 * V.  Consecutive threads take consecutive channel
// vectors of the same pixels (coalesced 16-byte accesses); padding reads zero.
// Weights in [3][3][C].
template <int STRIDE, int V>
__global__ __launch_bounds__(256) void dwconv3x3_kernel(const bf16* __restrict__ x, int N, int H, int W, int C,
                                                        const bf16* __restrict__ w, const float* __restrict__ scale,
                                                        const float* __restrict__ shift, int act,
                                                        bf16* __restrict__ y, int Ho, int Wo) {
  constexpr int COLS = (V - 1) * STRIDE + 3;  // input columns a row of the window spans
  const int CV = C >> 3;
  const int segs = (Wo + V - 1) / V;
  const long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  const long total = (long)N * Ho * segs * CV;
  if (idx >= total) return;
  const int cv = (int)(idx % CV);
  long t = idx / CV;
  const int seg = (int)(t % segs);
  t /= segs;
  const int ho = (int)(t % Ho);
  const int n = (int)(t / Ho);
  const int wo0 = seg * V;
  const int wi0 = wo0 * STRIDE - 1;

  bf16x8 wv[9];
#pragma unroll
  for (int k = 0; k < 9; ++k) wv[k] = ld8(w + k * C + cv * 8);
  float acc[V][8];
#pragma unroll
  for (int v = 0; v < V; ++v)
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[v][e] = 0.f;

#pragma unroll
  for (int r = 0; r < 3; ++r) {
    const int hi = ho * STRIDE - 1 + r;
    if ((unsigned)hi >= (unsigned)H) continue;
    const bf16* xrow = x + (((long)n * H + hi) * W) * C + cv * 8;
#pragma unroll
    for (int c = 0; c < COLS; ++c) {
      const int wi = wi0 + c;
      const bf16x8 xv = (unsigned)wi < (unsigned)W ? ld8(xrow + (long)wi * C) : bf16x8{};
      // outputs v whose window column s = c - v*STRIDE lies in 0..2
#pragma unroll
      for (int v = 0; v < V; ++v) {
        const int s = c - v * STRIDE;
        if (s < 0 || s > 2) continue;
#pragma unroll
        for (int e = 0; e < 8; ++e) acc[v][e] += (float)xv[e] * (float)wv[r * 3 + s][e];
      }
    }
  }
  const f32x4* sc = reinterpret_cast<const f32x4*>(scale + cv * 8);
  const f32x4* sh = reinterpret_cast<const f32x4*>(shift + cv * 8);
  const f32x4 s0 = sc[0], s1 = sc[1], h0 = sh[0], h1 = sh[1];
  bf16* yrow = y + (((long)n * Ho + ho) * Wo) * C + cv * 8;
#pragma unroll
  for (int v = 0; v < V; ++v) {
    if (wo0 + v >= Wo) break;
    bf16x8 o;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      o[e] = (bf16)apply_act(acc[v][e] * s0[e] + h0[e], act);
      o[e + 4] = (bf16)apply_act(acc[v][e + 4] * s1[e] + h1[e], act);
    }
    st8(yrow + (long)(wo0 + v) * C, o);
  }
}

template <int STRIDE, int V>
static void dw_launch(const bf16* x, int N, int H, int W, int C, const bf16* w, const float* scale,
                      const float* shift, int act, bf16* y, int Ho, int Wo, hipStream_t st) {
  const long total = (long)N * Ho * ((Wo + V - 1) / V) * (C / 8);
  launch(dwconv3x3_kernel<STRIDE, V>, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, x, N, H,
                     W, C, w, scale, shift, act, y, Ho, Wo);
}

dstack_status launch_dwconv3x3(const bf16* x, int N, int H, int W, int C, const bf16* w_rsc, int stride,
                               const float* scale, const float* shift, int act, bf16* y, hipStream_t st) {
  DS_CHECK(C % 8 == 0, DSTACK_E_UNSUPPORTED, "dwconv3x3: C must be a multiple of 8");
  DS_CHECK(stride == 1 || stride == 2, DSTACK_E_UNSUPPORTED, "dwconv3x3: stride must be 1 or 2");
  DS_CHECK(N > 0 && H > 0 && W > 0, DSTACK_E_INVALID, "dwconv3x3: bad shape");
  DS_CHECK(scale && shift, DSTACK_E_INVALID, "dwconv3x3: scale and shift are required");
  const int Ho = out_dim(H, 3, stride, 1), Wo = out_dim(W, 3, stride, 1);
  // outputs per thread along W: 8 on stride-1 rows at least 28 wide with more
  // than 32 channels, else 4
  if (stride == 1) {
    if (Wo >= 28 && C > 32)
      dw_launch<1, 8>(x, N, H, W, C, w_rsc, scale, shift, act, y, Ho, Wo, st);
    else
      dw_launch<1, 4>(x, N, H, W, C, w_rsc, scale, shift, act, y, Ho, Wo, st);
  } else {
    dw_launch<2, 4>(x, N, H, W, C, w_rsc, scale, shift, act, y, Ho, Wo, st);
  }
  DS_HIP(hipGetLastError());
  return DSTACK_OK;
}

// ------------------------------------------------------------- pooling ----
__global__ __launch_bounds__(256) void maxpool_kernel(const bf16* __restrict__ x, int N, int H, int W, int C, int k,
                                                      int stride, int pad, bf16* __restrict__ y, int Ho, int Wo) {
  const int CV = C >> 3;
  long idx = (long)blockIdx.x * blockDim.x + threadIdx.x;
  long total = (long)N * Ho * Wo * CV;
  if (idx >= total) return;
  int cv = (int)(idx % CV);
  long pix = idx / CV;
  int wo = (int)(pix % Wo);
  long t = pix / Wo;
  int ho = (int)(t % Ho);
  int n = (int)(t / Ho);
  float m[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) m[e] = -INFINITY;
  for (int r = 0; r < k; ++r) {
    int hi = ho * stride - pad + r;
    if ((unsigned)hi >= (unsigned)H) continue;
    for (int s = 0; s < k; ++s) {
      int wi = wo * stride - pad + s;
      if ((unsigned)wi >= (unsigned)W) continue;
      bf16x8 v = ld8(x + (((long)n * H + hi) * W + wi) * C + cv * 8);
#pragma unroll
      for (int e = 0; e < 8; ++e) m[e] = fmaxf(m[e], (float)v[e]);
    }
  }
  bf16x8 o;
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = (bf16)m[e];
  st8(y + pix * C + cv * 8, o);
}

dstack_status launch_maxpool(const bf16* x, int N, int H, int W, int C, int k, int stride, int pad, bf16* y,
                             hipStream_t st) {
  DS_CHECK(C % 8 == 0, DSTACK_E_UNSUPPORTED, "maxpool: C must be a multiple of 8");
  DS_CHECK(k > 0 && stride > 0 && pad >= 0 && pad < k && N > 0 && H > 0 && W > 0, DSTACK_E_INVALID,
           "maxpool: bad shape");
  int Ho = out_dim(H, k, stride, pad), Wo = out_dim(W, k, stride, pad);
  DS_CHECK(Ho > 0 && Wo > 0, DSTACK_E_INVALID, "maxpool: empty output");
  long total = (long)N * Ho * Wo * (C / 8);
  launch(maxpool_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, x, N, H, W, C, k,
                     stride, pad, y, Ho, Wo);
  DS_HIP(hipGetLastError());
  return DSTACK_OK;
}

// Global average pool.  Block = 32 channel vectors (8 channels each) x 8
// position groups of one image: thread (g, v) sums positions g, g+8, ... of
// vector v (its loads independent and in flight together), fp32 partial sums
// are combined in LDS and thread g = 0 writes the mean.
__global__ __launch_bounds__(256) void avgpool_kernel(const bf16* __restrict__ x, int N, int HW, int C,
                                                      bf16* __restrict__ y) {
  __shared__ float part[8][32][9];  // [group][vector][8 sums + pad]
  const int CV = C >> 3;
  const int v = threadIdx.x & 31, g = threadIdx.x >> 5;
  const int cv = blockIdx.x * 32 + v, n = blockIdx.y;
  float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  if (cv < CV) {
    const bf16* p = x + (long)n * HW * C + cv * 8;
#pragma unroll 4
    for (int i = g; i < HW; i += 8) {
      const bf16x8 t = ld8(p + (long)i * C);
#pragma unroll
      for (int e = 0; e < 8; ++e) s[e] += (float)t[e];
    }
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) part[g][v][e] = s[e];
  __syncthreads();
  if (g != 0 || cv >= CV) return;
  const float inv = 1.0f / (float)HW;
  bf16x8 o;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    float t = 0.f;
#pragma unroll
    for (int k = 0; k < 8; ++k) t += part[k][v][e];
    o[e] = (bf16)(t * inv);
  }
  st8(y + (long)n * C + cv * 8, o);
}

dstack_status launch_avgpool(const bf16* x, int N, int H, int W, int C, bf16* y, hipStream_t st) {
  DS_CHECK(C % 8 == 0, DSTACK_E_UNSUPPORTED, "avgpool: C must be a multiple of 8");
  DS_CHECK(N > 0 && H > 0 && W > 0 && N <= 65535, DSTACK_E_INVALID, "avgpool: bad shape");
  launch(avgpool_kernel, dim3(ceil_div(C / 8, 32), N), dim3(256), 0, st, x, N, H * W, C, y);
  DS_HIP(hipGetLastError());
  return DSTACK_OK;
}

// -------------------------------------------------------------- probe ----
// Each one-wave block records the hardware XCC id and HW_ID register (CU,
// SH, SE fields) of the CU it ran on, then spins briefly so that the
// dispatcher spreads the blocks over every CU the stream's mask allows.
__global__ void probe_kernel(uint32_t* out, int n) {
  if (threadIdx.x == 0 && (int)blockIdx.x < n) {
    uint32_t xcc = __builtin_amdgcn_s_getreg((3 << 11) | (0 << 6) | 20);   // HW_REG_XCC_ID[3:0]
    uint32_t hw = __builtin_amdgcn_s_getreg((31 << 11) | (0 << 6) | 4);    // HW_REG_HW_ID
    out[2 * blockIdx.x] = xcc;
    out[2 * blockIdx.x + 1] = hw;
    long t0 = clock64();
    while (clock64() - t0 < 20000) {
    }
  }
}

dstack_status launch_probe(uint32_t* d_out, int n_blocks, hipStream_t st) {
  launch(probe_kernel, dim3(n_blocks), dim3(64), 0, st, d_out, n_blocks);
  DS_HIP(hipGetLastError());
  return DSTACK_OK;
}

}  // namespace dstack
