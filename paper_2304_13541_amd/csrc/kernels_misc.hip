// Memory-bound kernels of the hot path: depthwise 3x3 convolution, small-batch
// fully-connected layers, pooling and input packing, plus the LSTM step.
// In the paper's terms (Sec. 4.1) these are the low arithmetic-intensity
// kernels: they are written for coalesced 16-byte accesses along the channel
// (NHWC) or feature axis and wave-level reductions, not for matrix cores --
// except the LSTM recurrence, whose [4H x H] x [H x B] product per step is
// small enough to sit on MFMA while its time goes to streaming W_hh.
#include <mutex>

#include "common.hpp"

namespace dstack {

__device__ __forceinline__ bf16x8 ld8(const bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }
__device__ __forceinline__ void st8(bf16* p, bf16x8 v) { *reinterpret_cast<bf16x8*>(p) = v; }

// ------------------------------------------------------------ depthwise ----
// One thread per (output pixel, 8-channel group).  Weights in [3][3][C].
template <int STRIDE>
__global__ __launch_bounds__(256) void dwconv3x3_kernel(const bf16* __restrict__ x, int N, int H, int W, int C,
                                                        const bf16* __restrict__ w, const float* __restrict__ scale,
                                                        const float* __restrict__ shift, int act,
                                                        bf16* __restrict__ y, int Ho, int Wo) {
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
  float acc[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
#pragma unroll
  for (int r = 0; r < 3; ++r) {
    int hi = ho * STRIDE - 1 + r;
    if ((unsigned)hi >= (unsigned)H) continue;
#pragma unroll
    for (int s = 0; s < 3; ++s) {
      int wi = wo * STRIDE - 1 + s;
      if ((unsigned)wi >= (unsigned)W) continue;
      bf16x8 xv = ld8(x + (((long)n * H + hi) * W + wi) * C + cv * 8);
      bf16x8 wv = ld8(w + (r * 3 + s) * C + cv * 8);
#pragma unroll
      for (int e = 0; e < 8; ++e) acc[e] += (float)xv[e] * (float)wv[e];
    }
  }
  const f32x4* sc = reinterpret_cast<const f32x4*>(scale + cv * 8);
  const f32x4* sh = reinterpret_cast<const f32x4*>(shift + cv * 8);
  f32x4 s0 = sc[0], s1 = sc[1], h0 = sh[0], h1 = sh[1];
  bf16x8 o;
#pragma unroll
  for (int e = 0; e < 4; ++e) {
    o[e] = (bf16)apply_act(acc[e] * s0[e] + h0[e], act);
    o[e + 4] = (bf16)apply_act(acc[e + 4] * s1[e] + h1[e], act);
  }
  st8(y + pix * C + cv * 8, o);
}

dstack_status launch_dwconv3x3(const bf16* x, int N, int H, int W, int C, const bf16* w_rsc, int stride,
                               const float* scale, const float* shift, int act, bf16* y, hipStream_t st) {
  DS_CHECK(C % 8 == 0, DSTACK_E_UNSUPPORTED, "dwconv3x3: C must be a multiple of 8");
  DS_CHECK(stride == 1 || stride == 2, DSTACK_E_UNSUPPORTED, "dwconv3x3: stride must be 1 or 2");
  DS_CHECK(N > 0 && H > 0 && W > 0, DSTACK_E_INVALID, "dwconv3x3: bad shape");
  int Ho = out_dim(H, 3, stride, 1), Wo = out_dim(W, 3, stride, 1);
  long total = (long)N * Ho * Wo * (C / 8);
  dim3 grid((unsigned)((total + 255) / 256));
  if (stride == 1)
    hipLaunchKernelGGL(dwconv3x3_kernel<1>, grid, dim3(256), 0, st, x, N, H, W, C, w_rsc, scale, shift, act, y, Ho, Wo);
  else
    hipLaunchKernelGGL(dwconv3x3_kernel<2>, grid, dim3(256), 0, st, x, N, H, W, C, w_rsc, scale, shift, act, y, Ho, Wo);
  DS_HIP(hipGetLastError());
  return DSTACK_OK;
}

// ------------------------------------------------------------------ FC ----
// One wave per R output features.  Lanes stride the input features 8 at a
// time (16-byte loads of the weight rows), every lane keeps R x BMAX partial
// dot products, and a butterfly over the 64 lanes finishes each one.
template <int R, int BMAX>
__global__ __launch_bounds__(256) void fc_kernel(const bf16* __restrict__ x, int B, int I, const bf16* __restrict__ w,
                                                 const float* __restrict__ bias, int O, int act, void* y, int out_f32) {
  const int lane = threadIdx.x & 63;
  const int o0 = ((blockIdx.x * blockDim.x + threadIdx.x) >> 6) * R;
  if (o0 >= O) return;
  float acc[R][BMAX];
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int b = 0; b < BMAX; ++b) acc[r][b] = 0.f;
  for (int i = lane * 8; i < I; i += 512) {
    bf16x8 wv[R];
#pragma unroll
    for (int r = 0; r < R; ++r) wv[r] = (o0 + r < O) ? ld8(w + (long)(o0 + r) * I + i) : bf16x8{};
#pragma unroll
    for (int b = 0; b < BMAX; ++b) {
      if (b < B) {
        bf16x8 xv = ld8(x + (long)b * I + i);
#pragma unroll
        for (int r = 0; r < R; ++r)
#pragma unroll
          for (int e = 0; e < 8; ++e) acc[r][b] += (float)wv[r][e] * (float)xv[e];
      }
    }
  }
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int b = 0; b < BMAX; ++b) {
      float v = acc[r][b];
#pragma unroll
      for (int off = 32; off >= 1; off >>= 1) v += __shfl_xor(v, off, 64);
      acc[r][b] = v;
    }
  // lane j writes entry (r, b) with j = r * BMAX + b
#pragma unroll
  for (int r = 0; r < R; ++r)
#pragma unroll
    for (int b = 0; b < BMAX; ++b) {
      if (lane == r * BMAX + b && b < B && o0 + r < O) {
        float v = apply_act(acc[r][b] + (bias ? bias[o0 + r] : 0.f), act);
        long idx = (long)b * O + o0 + r;
        if (out_f32)
          reinterpret_cast<float*>(y)[idx] = v;
        else
          reinterpret_cast<bf16*>(y)[idx] = (bf16)v;
      }
    }
}

template <int R, int BMAX>
static void fc_launch(const bf16* x, int B, int I, const bf16* w, const float* bias, int O, int act, void* y,
                      bool f32, hipStream_t st) {
  static_assert(R * BMAX <= 64, "one lane per output entry");
  int waves = ceil_div(O, R);
  hipLaunchKernelGGL((fc_kernel<R, BMAX>), dim3(ceil_div(waves, 4)), dim3(256), 0, st, x, B, I, w, bias, O, act, y,
                     f32 ? 1 : 0);
}

dstack_status launch_fc(const bf16* x, int B, int I, const bf16* w, const float* bias, int O, int act, void* y,
                        bool out_fp32, hipStream_t st) {
  DS_CHECK(B >= 1 && B <= 32, DSTACK_E_UNSUPPORTED, "fc: batch must be 1..32");
  DS_CHECK(I % 8 == 0 && I > 0 && O > 0, DSTACK_E_UNSUPPORTED, "fc: I must be a positive multiple of 8");
  if (B <= 8)
    fc_launch<8, 8>(x, B, I, w, bias, O, act, y, out_fp32, st);
  else if (B <= 16)
    fc_launch<4, 16>(x, B, I, w, bias, O, act, y, out_fp32, st);
  else
    fc_launch<2, 32>(x, B, I, w, bias, O, act, y, out_fp32, st);
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
  hipLaunchKernelGGL(maxpool_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, st, x, N, H, W, C, k,
                     stride, pad, y, Ho, Wo);
  DS_HIP(hipGetLastError());
  return DSTACK_OK;
}

// Global average pool: one thread per (image, 8-channel group), fp32 sum.
__global__ __launch_bounds__(256) void avgpool_kernel(const bf16* __restrict__ x, int N, int HW, int C,
                                                      bf16* __restrict__ y) {
  const int CV = C >> 3;
  int idx = blockIdx.x * blockDim.x + threadIdx.x;
  if (idx >= N * CV) return;
  int cv = idx % CV, n = idx / CV;
  float s[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
  const bf16* p = x + (long)n * HW * C + cv * 8;
  for (int i = 0; i < HW; ++i) {
    bf16x8 v = ld8(p + (long)i * C);
#pragma unroll
    for (int e = 0; e < 8; ++e) s[e] += (float)v[e];
  }
  float inv = 1.0f / (float)HW;
  bf16x8 o;
#pragma unroll
  for (int e = 0; e < 8; ++e) o[e] = (bf16)(s[e] * inv);
  st8(y + (long)n * C + cv * 8, o);
}

dstack_status launch_avgpool(const bf16* x, int N, int H, int W, int C, bf16* y, hipStream_t st) {
  DS_CHECK(C % 8 == 0, DSTACK_E_UNSUPPORTED, "avgpool: C must be a multiple of 8");
  DS_CHECK(N > 0 && H > 0 && W > 0, DSTACK_E_INVALID, "avgpool: bad shape");
  int total = N * (C / 8);
  hipLaunchKernelGGL(avgpool_kernel, dim3(ceil_div(total, 256)), dim3(256), 0, st, x, N, H * W, C, y);
  DS_HIP(hipGetLastError());
  return DSTACK_OK;
}

// Input packing: [npix][C] -> [npix][8] with zero channels C..7 (C <= 8).
__global__ __launch_bounds__(256) void pack_c8_kernel(const bf16* __restrict__ x, long npix, int C,
                                                      bf16* __restrict__ y) {
  long p = (long)blockIdx.x * blockDim.x + threadIdx.x;
  if (p >= npix) return;
  bf16x8 o = {};
  for (int c = 0; c < C; ++c) o[c] = x[p * C + c];
  st8(y + p * 8, o);
}

dstack_status launch_pack_c8(const bf16* x, int npix, int C, bf16* y, hipStream_t st) {
  DS_CHECK(C >= 1 && C <= 8 && npix > 0, DSTACK_E_INVALID, "pack: bad shape");
  hipLaunchKernelGGL(pack_c8_kernel, dim3(ceil_div(npix, 256)), dim3(256), 0, st, x, (long)npix, C, y);
  DS_HIP(hipGetLastError());
  return DSTACK_OK;
}

// ----------------------------------------------------------- LSTM step ----
// gates[b][g*H + j] = gx_t[b][g*H + j] + sum_k W_hh[g*H + j][k] * h_prev[b][k]
// then c = f*c + i*g~, h = o*tanh(c) (gate order i, f, g, o).
// Block = 4 waves on 16 hidden units; wave w owns units j0 + 4w .. +3 and
// all four gates of them: the 16 MFMA rows are (gate, unit) = (row/4, row%4),
// so the 16x16x32 result gives lane l gate l/16 of units 0..3 for batch
// column l%16.  h_prev [B][H] is staged once per block in LDS.  The four
// gates of one (unit, batch) are regrouped through LDS for the cell update.
constexpr int LSTM_UNITS_PER_BLOCK = 16;

__global__ __launch_bounds__(256) void lstm_step_kernel(const float* __restrict__ gx, const bf16* __restrict__ whh,
                                                        const bf16* __restrict__ hprev, float* __restrict__ c,
                                                        bf16* __restrict__ hnext, float* __restrict__ hf32, int B,
                                                        int H, int first) {
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  bf16* hs = reinterpret_cast<bf16*>(smem);                              // [32][H + 8]
  const int HP = H + 8;
  float* gs = reinterpret_cast<float*>(smem + (size_t)32 * HP * sizeof(bf16)); // [4 waves][2][4 gates][4 units][16]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int j0 = blockIdx.x * LSTM_UNITS_PER_BLOCK + wave * 4;
  const int nmt = (B + 15) / 16;

  f32x4 acc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
  if (!first) {
    // stage h_prev rows 0..nmt*16-1 (zero beyond B)
    const int chunks = H / 8;
    for (int q = tid; q < nmt * 16 * chunks; q += 256) {
      int b = q / chunks, k = (q % chunks) * 8;
      bf16x8 v = b < B ? ld8(hprev + (long)b * H + k) : bf16x8{};
      st8(hs + b * HP + k, v);
    }
    __syncthreads();
    const int row = lane & 15;
    const bf16* wrow = whh + (long)((row >> 2) * H + j0 + (row & 3)) * H;
    const int koff = (lane >> 4) * 8;
    for (int k = 0; k < H; k += 32) {
      bf16x8 a = ld8(wrow + k + koff);
      for (int mt = 0; mt < nmt; ++mt) {
        bf16x8 bv = *reinterpret_cast<const bf16x8*>(hs + (mt * 16 + (lane & 15)) * HP + k + koff);
        acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, bv, acc[mt], 0, 0, 0);
      }
    }
  }
  // regroup: gs[wave][mt][g][u][b16]
  float* gw = gs + wave * (2 * 4 * 4 * 16);
  {
    const int g = lane >> 4, bcol = lane & 15;
    for (int mt = 0; mt < nmt; ++mt)
#pragma unroll
      for (int u = 0; u < 4; ++u) gw[((mt * 4 + g) * 4 + u) * 16 + bcol] = acc[mt][u];
  }
  __syncthreads();
  {
    const int u = lane >> 4, bcol = lane & 15;
    const int j = j0 + u;
    for (int mt = 0; mt < nmt; ++mt) {
      const int b = mt * 16 + bcol;
      if (b >= B) continue;
      const float* gxb = gx + (long)b * 4 * H;
      float gi = gw[((mt * 4 + 0) * 4 + u) * 16 + bcol] + gxb[0 * H + j];
      float gf = gw[((mt * 4 + 1) * 4 + u) * 16 + bcol] + gxb[1 * H + j];
      float gg = gw[((mt * 4 + 2) * 4 + u) * 16 + bcol] + gxb[2 * H + j];
      float go = gw[((mt * 4 + 3) * 4 + u) * 16 + bcol] + gxb[3 * H + j];
      float ig = 1.f / (1.f + __expf(-gi));
      float fg = 1.f / (1.f + __expf(-gf));
      float gt = tanhf(gg);
      float og = 1.f / (1.f + __expf(-go));
      float cp = first ? 0.f : c[(long)b * H + j];
      float cn = fg * cp + ig * gt;
      float hn = og * tanhf(cn);
      c[(long)b * H + j] = cn;
      hnext[(long)b * H + j] = (bf16)hn;
      if (hf32) hf32[(long)b * H + j] = hn;
    }
  }
}

size_t lstm_step_lds_bytes(int H) { return (size_t)32 * (H + 8) * sizeof(bf16) + 4 * 2 * 4 * 4 * 16 * sizeof(float); }

dstack_status launch_lstm_step(const float* gx_t, const bf16* w_hh, const bf16* h_prev, float* c, bf16* h_next,
                               float* h_f32, int B, int H, bool first, hipStream_t st) {
  DS_CHECK(B >= 1 && B <= 32, DSTACK_E_UNSUPPORTED, "lstm: batch must be 1..32");
  // the depth loop steps by 32 and each block owns 16 units
  DS_CHECK(H % 32 == 0 && H >= 32, DSTACK_E_UNSUPPORTED, "lstm: H must be a multiple of 32");
  size_t lds = lstm_step_lds_bytes(H);
  DS_CHECK(lds <= 160 * 1024, DSTACK_E_UNSUPPORTED, "lstm: H too large for the LDS staging of h");
  static std::once_flag once;
  std::call_once(once, [] {
    (void)hipFuncSetAttribute((const void*)lstm_step_kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                              160 * 1024);
  });
  hipLaunchKernelGGL(lstm_step_kernel, dim3(H / LSTM_UNITS_PER_BLOCK), dim3(256), lds, st, gx_t, w_hh, h_prev, c,
                     h_next, h_f32, B, H, first ? 1 : 0);
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
  hipLaunchKernelGGL(probe_kernel, dim3(n_blocks), dim3(64), 0, st, d_out, n_blocks);
  DS_HIP(hipGetLastError());
  return DSTACK_OK;
}

}  // namespace dstack
