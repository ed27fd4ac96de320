// Weight-streaming kernels: small-batch fully connected layers and the LSTM
// recurrence.  Both read a large weight matrix once per call while the
// activations (a handful of rows) stay in L2, so they are bound by HBM (or
// the Infinity Cache) and by load latency, not by arithmetic (the LSTM is the
// low arithmetic-intensity example of the compute- vs memory-bound kernel table, Sec. 4.1).  Both split the
// reduction dimension over the four waves of a block, issue a wave's weight
// loads before consuming any of them, and combine partial sums in LDS.
#include "common.hpp"

namespace dstack {

namespace {

__device__ __forceinline__ bf16x8 ld8(const bf16* p) { return *reinterpret_cast<const bf16x8*>(p); }

}  // namespace

// ------------------------------------------------------------------ FC ----
// y[b][o] = act(sum_i x[b][i] * w[o][i] + bias[o]) for a batch of 1..32.
// A batch-B layer does B multiply-adds per weight element, which for B >= 8
// outruns the vector ALUs at HBM speed, so the product runs on
// v_mfma_f32_16x16x32_bf16: A = 16 weight rows (row o0 + lane % 16, depth
// 8 * (lane / 16) .. + 8 of each 32-deep step), B = the batch as 16 columns
// (NT tiles of 16).  Block (o-tile of 16 rows, depth split): its depth steps
// are dealt to the 4 waves in contiguous runs; a wave streams its run in
// chunks of CH steps, loading the next chunk before multiplying the current
// one.  Rows past O and batch columns past B read a clamped in-bounds row and
// are dropped at the end; depth past I reads nothing.  The 4 waves' tiles are
// summed through LDS; with one split the block applies bias and activation,
// otherwise it stores fp32 partial sums [split][B][O] for fc_reduce_kernel.
constexpr int FC_CH = 8;

template <int NT>
__device__ __forceinline__ void fc_load(const bf16* wrow, const bf16* const* xrow, int st, int ke, int I, int g,
                                        bf16x8 (&a)[FC_CH], bf16x8 (&bv)[FC_CH][NT]) {
#pragma unroll
  for (int j = 0; j < FC_CH; ++j) {
    const int k = (st + j) * 32 + g * 8;
    const bool in = st + j < ke && k < I;
    a[j] = in ? ld8(wrow + k) : bf16x8{};
#pragma unroll
    for (int t = 0; t < NT; ++t) bv[j][t] = in ? ld8(xrow[t] + k) : bf16x8{};
  }
}

template <int NT>
__device__ __forceinline__ void fc_mma(const bf16x8 (&a)[FC_CH], const bf16x8 (&bv)[FC_CH][NT], f32x4 (&acc)[NT]) {
#pragma unroll
  for (int j = 0; j < FC_CH; ++j)
#pragma unroll
    for (int t = 0; t < NT; ++t) acc[t] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[j], bv[j][t], acc[t], 0, 0, 0);
}

template <int NT>
__global__ __launch_bounds__(256) void fc_kernel(const bf16* __restrict__ x, int B, int I, const bf16* __restrict__ w,
                                                 const float* __restrict__ bias, int O, int act, void* y, int out_f32,
                                                 float* __restrict__ part, int steps_per_split) {
  __shared__ float red[4][NT][16][16];  // [wave][batch tile][row][batch column]
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int g = lane >> 4;
  const int o0 = blockIdx.x * 16, split = blockIdx.y;
  const int nks = (I + 31) >> 5;
  const int kb0 = split * steps_per_split, kb1 = min(nks, kb0 + steps_per_split);
  const int per = (kb1 - kb0 + 3) >> 2;
  const int ks = kb0 + wave * per, ke = min(kb1, ks + per);

  const bf16* wrow = w + (long)min(o0 + (lane & 15), O - 1) * I;
  const bf16* xrow[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) xrow[t] = x + (long)min(t * 16 + (lane & 15), B - 1) * I;

  f32x4 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (ks < ke) {
    bf16x8 a0[FC_CH], b0[FC_CH][NT], a1[FC_CH], b1[FC_CH][NT];
    fc_load<NT>(wrow, xrow, ks, ke, I, g, a0, b0);
    for (int st = ks; st < ke; st += 2 * FC_CH) {
      if (st + FC_CH < ke) fc_load<NT>(wrow, xrow, st + FC_CH, ke, I, g, a1, b1);
      fc_mma<NT>(a0, b0, acc);
      if (st + 2 * FC_CH < ke) fc_load<NT>(wrow, xrow, st + 2 * FC_CH, ke, I, g, a0, b0);
      if (st + FC_CH < ke) fc_mma<NT>(a1, b1, acc);
    }
  }
  // C layout: lane holds rows 4 * (lane / 16) + i, batch column lane % 16
#pragma unroll
  for (int t = 0; t < NT; ++t)
#pragma unroll
    for (int i = 0; i < 4; ++i) red[wave][t][4 * g + i][lane & 15] = acc[t][i];
  __syncthreads();
  for (int e = threadIdx.x; e < NT * 256; e += 256) {
    const int row = e & 15, col = (e >> 4) & 15, t = e >> 8;  // row fastest: consecutive o per store
    const int o = o0 + row, b = t * 16 + col;
    if (o >= O || b >= B) continue;
    float v = red[0][t][row][col] + red[1][t][row][col] + red[2][t][row][col] + red[3][t][row][col];
    if (gridDim.y > 1) {
      part[((long)split * B + b) * O + o] = v;
      continue;
    }
    v = apply_act(v + (bias ? bias[o] : 0.f), act);
    if (out_f32)
      reinterpret_cast<float*>(y)[(long)b * O + o] = v;
    else
      reinterpret_cast<bf16*>(y)[(long)b * O + o] = (bf16)v;
  }
}

__global__ __launch_bounds__(256) void fc_reduce_kernel(const float* __restrict__ part, int splits, int B, int O,
                                                        const float* __restrict__ bias, int act, void* y,
                                                        int out_f32) {
  const int e = blockIdx.x * 256 + threadIdx.x;  // b * O + o
  if (e >= B * O) return;
  float v = 0.f;
  for (int s = 0; s < splits; ++s) v += part[(long)s * B * O + e];
  v = apply_act(v + (bias ? bias[e % O] : 0.f), act);
  if (out_f32)
    reinterpret_cast<float*>(y)[e] = v;
  else
    reinterpret_cast<bf16*>(y)[e] = (bf16)v;
}

// Depth split: double while the grid is below 2 blocks per CU and every block
// keeps at least 16 depth steps (4 per wave), up to 16 splits.
static int fc_splits(int I, int O, int n_cu) {
  const int tiles = (O + 15) / 16, nks = (I + 31) / 32;
  int s = 1;
  while (s < 16 && tiles * s < 2 * n_cu && nks / (2 * s) >= 16) s *= 2;
  return s;
}

size_t fc_workspace_bytes(int B, int I, int O, int n_cu) {
  const int s = fc_splits(I, O, n_cu > 0 ? n_cu : 256);
  return s > 1 ? (size_t)s * B * O * sizeof(float) : 0;
}

dstack_status launch_fc(const bf16* x, int B, int I, const bf16* w, const float* bias, int O, int act, void* y,
                        bool out_fp32, int n_cu, float* ws, size_t ws_bytes, hipStream_t st) {
  DS_CHECK(B >= 1 && B <= 32, DSTACK_E_UNSUPPORTED, "fc: batch must be 1..32");
  DS_CHECK(I % 8 == 0 && I > 0 && O > 0, DSTACK_E_UNSUPPORTED, "fc: I must be a positive multiple of 8");
  DS_CHECK((long)O * I < (1L << 40) && (long)B * O < (1L << 30), DSTACK_E_UNSUPPORTED, "fc: too large");
  int s = fc_splits(I, O, n_cu > 0 ? n_cu : 256);
  while (s > 1 && (!ws || (size_t)s * B * O * sizeof(float) > ws_bytes)) s /= 2;
  const int nks = (I + 31) / 32;
  const int sps = (nks + s - 1) / s;
  s = (nks + sps - 1) / sps;  // no empty split
  dim3 grid((O + 15) / 16, s);
  const int f = out_fp32 ? 1 : 0;
  if (B <= 16)
    launch(fc_kernel<1>, grid, dim3(256), 0, st, x, B, I, w, bias, O, act, y, f, ws, sps);
  else
    launch(fc_kernel<2>, grid, dim3(256), 0, st, x, B, I, w, bias, O, act, y, f, ws, sps);
  DS_HIP(hipGetLastError());
  if (s > 1) {
    launch(fc_reduce_kernel, dim3((B * O + 255) / 256), dim3(256), 0, st, ws, s, B, O, bias, act, y, f);
    DS_HIP(hipGetLastError());
  }
  return DSTACK_OK;
}

// ----------------------------------------------------------- LSTM step ----
// gates[b][g*H + j] = gx_t[b][g*H + j] + sum_k W_hh[g*H + j][k] * h_prev[b][k],
// then c = f*c + i*g~, h = o*tanh(c) (gate order i, f, g, o; h_prev = 0 at t = 0).
// Block: 4 hidden units, i.e. the 16 rows (gate, unit) = (row / 4, row % 4)
// of one v_mfma_f32_16x16x32_bf16 A operand; wave w takes depth steps
// [w*KSW, (w+1)*KSW) of 32 and loads all of its W_hh fragments before the
// first MFMA.  B operand: h_prev rows (batch) read from L2.  Lane l ends with
// gate l/16 of units 0..3 for batch column l%16; the four waves' partial sums
// meet in LDS, where the 128 (unit, batch) cells are then updated by the
// first 128 threads.
template <int KSW>
__global__ __launch_bounds__(256) void lstm_step_kernel(const float* __restrict__ gx, const bf16* __restrict__ whh,
                                                        const bf16* __restrict__ hprev, float* __restrict__ c,
                                                        bf16* __restrict__ hnext, float* __restrict__ hf32, int B,
                                                        int H, int first) {
  __shared__ float gs[4][2][16][16];  // [wave][batch tile][row = gate*4 + unit][batch column]
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int j0 = blockIdx.x * 4;
  const int nmt = (B + 15) >> 4;
  const int nks = H >> 5;
  const int k0 = wave * KSW, k1 = min(nks, k0 + KSW);
  const int row = lane & 15;
  const int koff = (lane >> 4) * 8;
  // the cell threads fetch their input-projection gates and cell state now,
  // so that these loads overlap the recurrent product
  const int cu = tid >> 5, cb = tid & 31, cj = j0 + cu;  // unit, batch of a cell thread
  const bool cell = tid < 128 && cb < B;
  float gxv[4] = {0.f, 0.f, 0.f, 0.f}, cprev = 0.f;
  if (cell) {
#pragma unroll
    for (int g = 0; g < 4; ++g) gxv[g] = gx[(long)cb * 4 * H + g * H + cj];
    if (!first) cprev = c[(long)cb * H + cj];
  }

  f32x4 acc[2] = {f32x4{0.f, 0.f, 0.f, 0.f}, f32x4{0.f, 0.f, 0.f, 0.f}};
  if (!first && k0 < k1) {
    const bf16* wrow = whh + (long)((row >> 2) * H + j0 + (row & 3)) * H;
    bf16x8 a[KSW], bv[2][KSW];
#pragma unroll
    for (int s = 0; s < KSW; ++s) {
      const int k = (k0 + s) * 32 + koff;
      const bool in = k0 + s < k1;
      a[s] = in ? ld8(wrow + k) : bf16x8{};
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
        const int b = mt * 16 + (lane & 15);
        bv[mt][s] = (in && mt < nmt && b < B) ? ld8(hprev + (long)b * H + k) : bf16x8{};
      }
    }
#pragma unroll
    for (int s = 0; s < KSW; ++s)
#pragma unroll
      for (int mt = 0; mt < 2; ++mt)
        if (mt < nmt) acc[mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[s], bv[mt][s], acc[mt], 0, 0, 0);
  }
  // C layout: lane holds rows 4*(lane/16) + i, column lane%16
#pragma unroll
  for (int mt = 0; mt < 2; ++mt)
#pragma unroll
    for (int i = 0; i < 4; ++i) gs[wave][mt][4 * (lane >> 4) + i][lane & 15] = acc[mt][i];
  __syncthreads();
  if (cell) {
    const int mt = cb >> 4, bc = cb & 15;
    float g4[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int r = g * 4 + cu;
      g4[g] = gs[0][mt][r][bc] + gs[1][mt][r][bc] + gs[2][mt][r][bc] + gs[3][mt][r][bc] + gxv[g];
    }
    const float ig = 1.f / (1.f + __expf(-g4[0]));
    const float fg = 1.f / (1.f + __expf(-g4[1]));
    const float gt = tanhf(g4[2]);
    const float og = 1.f / (1.f + __expf(-g4[3]));
    const float cn = fg * cprev + ig * gt;
    const float hn = og * tanhf(cn);
    c[(long)cb * H + cj] = cn;
    hnext[(long)cb * H + cj] = (bf16)hn;
    if (hf32) hf32[(long)cb * H + cj] = hn;
  }
}

dstack_status launch_lstm_step(const float* gx_t, const bf16* w_hh, const bf16* h_prev, float* c, bf16* h_next,
                               float* h_f32, int B, int H, bool first, hipStream_t st) {
  DS_CHECK(B >= 1 && B <= 32, DSTACK_E_UNSUPPORTED, "lstm: batch must be 1..32");
  // depth is consumed in steps of 32; a block owns 4 hidden units
  DS_CHECK(H % 32 == 0 && H >= 32 && H <= 2048, DSTACK_E_UNSUPPORTED, "lstm: H must be a multiple of 32, <= 2048");
  const int nks = H / 32, ksw = (nks + 3) / 4;
  dim3 grid(H / 4), blk(256);
  const int f = first ? 1 : 0;
  if (ksw <= 2)
    launch(lstm_step_kernel<2>, grid, blk, 0, st, gx_t, w_hh, h_prev, c, h_next, h_f32, B, H, f);
  else if (ksw <= 4)
    launch(lstm_step_kernel<4>, grid, blk, 0, st, gx_t, w_hh, h_prev, c, h_next, h_f32, B, H, f);
  else if (ksw <= 8)
    launch(lstm_step_kernel<8>, grid, blk, 0, st, gx_t, w_hh, h_prev, c, h_next, h_f32, B, H, f);
  else
    launch(lstm_step_kernel<16>, grid, blk, 0, st, gx_t, w_hh, h_prev, c, h_next, h_f32, B, H, f);
  DS_HIP(hipGetLastError());
  return DSTACK_OK;
}

}  // namespace dstack
