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
// PK: the weights come in MFMA fragment order (a model's FC layers, packed
// at load): row tile ot and depth step s form a 16 x 32 block at
// ((ot * ceil(I/32) + s) * 16 + r) * 32, zero past O and I, so that a wave's
// load of a step reads 1 KB of consecutive bytes rather than 64-byte pieces
// of 16 rows.
constexpr int FC_CH = 8;

template <int NT, bool PK>
__device__ __forceinline__ void fc_load(const bf16* wrow, const bf16* const* xrow, int st, int ke, int I, int g,
                                        bf16x8 (&a)[FC_CH], bf16x8 (&bv)[FC_CH][NT]) {
#pragma unroll
  for (int j = 0; j < FC_CH; ++j) {
    const int k = (st + j) * 32 + g * 8;
    const bool in = st + j < ke && k < I;
    a[j] = in ? ld8(PK ? wrow + (long)(st + j) * 512 : wrow + k) : bf16x8{};
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

template <int NT, bool PK>
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

  // the lane's weight row (PK: its row and depth quarter of the tile's first step)
  const bf16* wrow = PK ? w + ((long)blockIdx.x * nks * 16 + (lane & 15)) * 32 + g * 8
                        : w + (long)min(o0 + (lane & 15), O - 1) * I;
  const bf16* xrow[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) xrow[t] = x + (long)min(t * 16 + (lane & 15), B - 1) * I;

  f32x4 acc[NT];
#pragma unroll
  for (int t = 0; t < NT; ++t) acc[t] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (ks < ke) {
    bf16x8 a0[FC_CH], b0[FC_CH][NT], a1[FC_CH], b1[FC_CH][NT];
    fc_load<NT, PK>(wrow, xrow, ks, ke, I, g, a0, b0);
    for (int st = ks; st < ke; st += 2 * FC_CH) {
      if (st + FC_CH < ke) fc_load<NT, PK>(wrow, xrow, st + FC_CH, ke, I, g, a1, b1);
      fc_mma<NT>(a0, b0, acc);
      if (st + 2 * FC_CH < ke) fc_load<NT, PK>(wrow, xrow, st + 2 * FC_CH, ke, I, g, a0, b0);
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

// Depth split: double while the grid has fewer blocks than the CUs and every
// block keeps at least 96 depth steps, up to 16 splits.  The split costs a
// second launch (the reduction), which only a long depth on a grid that
// leaves CUs idle repays.  Measured on MI355X (128 CUs, B = 8): 25088 -> 40
// (3 row tiles) 36.5 us unsplit, 10.0 us in 8; 25088 -> 1000 (63 tiles)
// 37.6 us unsplit, 23.2 us in 2; but VGG-19's 4096 -> 1000 (128 steps), and
// ResNet-50's and MobileNetV2's classifiers (64 and 40 steps), ran fastest
// unsplit, as did VGG-19's 25088 -> 4096 (256 tiles).
static int fc_splits(int I, int O, int n_cu) {
  const int tiles = (O + 15) / 16, nks = (I + 31) / 32;
  int s = 1;
  while (s < 16 && tiles * s < n_cu && nks / (2 * s) >= 96) s *= 2;
  return s;
}

size_t fc_workspace_bytes(int B, int I, int O, int n_cu) {
  const int s = fc_splits(I, O, n_cu > 0 ? n_cu : 256);
  return s > 1 ? (size_t)s * B * O * sizeof(float) : 0;
}

dstack_status launch_fc(const bf16* x, int B, int I, const bf16* w, const float* bias, int O, int act, void* y,
                        bool out_fp32, int n_cu, float* ws, size_t ws_bytes, hipStream_t st, bool packed) {
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
  if (packed) {
    if (B <= 16)
      launch(fc_kernel<1, true>, grid, dim3(256), 0, st, x, B, I, w, bias, O, act, y, f, ws, sps);
    else
      launch(fc_kernel<2, true>, grid, dim3(256), 0, st, x, B, I, w, bias, O, act, y, f, ws, sps);
  } else if (B <= 16) {
    launch(fc_kernel<1, false>, grid, dim3(256), 0, st, x, B, I, w, bias, O, act, y, f, ws, sps);
  } else {
    launch(fc_kernel<2, false>, grid, dim3(256), 0, st, x, B, I, w, bias, O, act, y, f, ws, sps);
  }
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
// Operands in MFMA fragment order, so that every wave load reads 1 KB of
// consecutive bytes (whole cache lines) rather than 16 half lines of 16
// different rows:
//  - W_hh packed once per layer run: row tile rt (the 16 rows (gate, unit) =
//    (r / 4, 4 rt + r % 4) of units 4rt .. 4rt+3) and depth step s (32 deep)
//    form a 16 x 32 block at ((rt * H/32 + s) * 16 + r) * 32;
//  - h(t-1) as written by the previous step: depth step s of batch row b at
//    (s * B + b) * 32.
// Block: U row tiles, i.e. 4U hidden units j0 .. j0 + 4U - 1.  Wave w takes
// depth steps [w*KSW, (w+1)*KSW) for all U row tiles and loads all of its
// W_hh and h fragments before the first MFMA.  Lane l ends with gate l/16 of
// a row tile's units for batch column l%16; the four waves' partial sums
// meet in LDS, where the 4U x B (unit, batch) cells are then updated, 256
// threads striding over them; each cell writes h in bf16 both row-major (the
// layer's output) and packed (the next step's operand), c in fp32.
// Every block reads all of h(t-1) (B x H) besides its 16U rows of W_hh, so U
// sets the step's L2 -> CU bytes: larger U reads h fewer times but leaves
// fewer blocks for the CUs.  The per-row sums (waves added in order 0..3,
// then the input projection) do not depend on U.
__global__ __launch_bounds__(256) void lstm_pack_whh_kernel(const bf16* __restrict__ w, bf16* __restrict__ wp,
                                                            int H) {
  const long v = (long)blockIdx.x * 256 + threadIdx.x;  // 16-byte vector of wp
  if (v >= (long)H * H / 2) return;                     // 4H x H elements, 8 per vector
  const int nks = H >> 5;
  const int q = (int)(v & 3);  // which 8 of the 32 depth values
  const int r = (int)((v >> 2) & 15);
  const long ts = v >> 6;  // rt * nks + s
  const int rt = (int)(ts / nks), st = (int)(ts - (long)rt * nks);
  const long src = (long)((r >> 2) * H + 4 * rt + (r & 3)) * H + st * 32 + q * 8;
  *reinterpret_cast<uint4*>(wp + v * 8) = *reinterpret_cast<const uint4*>(w + src);
}

template <int U, int KSW>
__global__ __launch_bounds__(256) void lstm_step_kernel(const float* __restrict__ gx, const bf16* __restrict__ wp,
                                                        const bf16* __restrict__ hp_prev, float* __restrict__ c,
                                                        bf16* __restrict__ hnext, bf16* __restrict__ hp_next,
                                                        float* __restrict__ hf32, int B, int H, int first) {
  // [wave][batch tile][row tile][row = gate*4 + unit][batch column]
  __shared__ float gs[4][2][U][16][16];
  constexpr int CPT = (128 * U + 255) / 256;  // cells per thread (a cell = (unit, batch), batch < 32)
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int rt0 = blockIdx.x * U, j0 = 4 * rt0;
  const int nmt = (B + 15) >> 4;
  const int nks = H >> 5;
  const int k0 = wave * KSW, k1 = min(nks, k0 + KSW);
  const int row = lane & 15;
  const int koff = (lane >> 4) * 8;
  // the cell threads fetch their input-projection gates and cell state now,
  // so that these loads overlap the recurrent product
  float gxv[CPT][4], cprev[CPT];
#pragma unroll
  for (int q = 0; q < CPT; ++q) {
    const int cell = tid + 256 * q, ul = cell >> 5, cb = cell & 31, cj = j0 + ul;
#pragma unroll
    for (int g = 0; g < 4; ++g) gxv[q][g] = 0.f;
    cprev[q] = 0.f;
    if (ul < 4 * U && cb < B) {
#pragma unroll
      for (int g = 0; g < 4; ++g) gxv[q][g] = gx[(long)cb * 4 * H + g * H + cj];
      if (!first) cprev[q] = c[(long)cb * H + cj];
    }
  }

  f32x4 acc[U][2];
#pragma unroll
  for (int u = 0; u < U; ++u) acc[u][0] = acc[u][1] = f32x4{0.f, 0.f, 0.f, 0.f};
  if (!first && k0 < k1) {
    bf16x8 a[U][KSW], bv[2][KSW];
#pragma unroll
    for (int s = 0; s < KSW; ++s) {
      const bool in = k0 + s < k1;
#pragma unroll
      for (int u = 0; u < U; ++u)
        a[u][s] = in ? ld8(wp + ((long)((rt0 + u) * nks + k0 + s) * 16 + row) * 32 + koff) : bf16x8{};
#pragma unroll
      for (int mt = 0; mt < 2; ++mt) {
        const int b = mt * 16 + (lane & 15);
        bv[mt][s] = (in && mt < nmt && b < B) ? ld8(hp_prev + ((long)(k0 + s) * B + b) * 32 + koff) : bf16x8{};
      }
    }
#pragma unroll
    for (int s = 0; s < KSW; ++s)
#pragma unroll
      for (int u = 0; u < U; ++u)
#pragma unroll
        for (int mt = 0; mt < 2; ++mt)
          if (mt < nmt) acc[u][mt] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[u][s], bv[mt][s], acc[u][mt], 0, 0, 0);
  }
  // C layout: lane holds rows 4*(lane/16) + i, column lane%16
#pragma unroll
  for (int u = 0; u < U; ++u)
#pragma unroll
    for (int mt = 0; mt < 2; ++mt)
#pragma unroll
      for (int i = 0; i < 4; ++i) gs[wave][mt][u][4 * (lane >> 4) + i][lane & 15] = acc[u][mt][i];
  __syncthreads();
#pragma unroll
  for (int q = 0; q < CPT; ++q) {
    const int cell = tid + 256 * q, ul = cell >> 5, cb = cell & 31, cj = j0 + ul;
    if (ul >= 4 * U || cb >= B) continue;
    const int mt = cb >> 4, bc = cb & 15, u = ul >> 2, cu = ul & 3;
    float g4[4];
#pragma unroll
    for (int g = 0; g < 4; ++g) {
      const int r = g * 4 + cu;
      g4[g] = gs[0][mt][u][r][bc] + gs[1][mt][u][r][bc] + gs[2][mt][u][r][bc] + gs[3][mt][u][r][bc] + gxv[q][g];
    }
    const float ig = 1.f / (1.f + __expf(-g4[0]));
    const float fg = 1.f / (1.f + __expf(-g4[1]));
    const float gt = tanhf(g4[2]);
    const float og = 1.f / (1.f + __expf(-g4[3]));
    const float cn = fg * cprev[q] + ig * gt;
    const float hn = og * tanhf(cn);
    c[(long)cb * H + cj] = cn;
    const bf16 hb = (bf16)hn;
    hnext[(long)cb * H + cj] = hb;
    hp_next[((long)(cj >> 5) * B + cb) * 32 + (cj & 31)] = hb;
    if (hf32) hf32[(long)cb * H + cj] = hn;
  }
}

// Groups of 4 units per block for a step on n_cu CUs: the U in {1, 2, 4}
// that gives the busiest CU the fewest bytes to load (its blocks' W_hh rows
// plus one h_prev each); ties go to the smaller U (more blocks).
int lstm_units_per_block(int B, int H, int n_cu) {
  const long cus = n_cu > 0 ? n_cu : 256;
  int best = 1;
  long best_bytes = -1;
  for (int u = 1; u <= 4; u *= 2) {
    const long blocks = H / (4 * u);
    const long per_cu = (blocks + cus - 1) / cus;
    const long bytes = per_cu * (16L * u * H * 2 + (long)B * H * 2);
    if (best_bytes < 0 || bytes < best_bytes) {
      best = u;
      best_bytes = bytes;
    }
  }
  return best;
}

template <int U>
static void launch_lstm_u(int ksw, dim3 grid, hipStream_t st, const float* gx_t, const bf16* wp, const bf16* hp_prev,
                          float* c, bf16* h_next, bf16* hp_next, float* h_f32, int B, int H, int f) {
  const dim3 blk(256);
  if (ksw <= 2)
    launch(lstm_step_kernel<U, 2>, grid, blk, 0, st, gx_t, wp, hp_prev, c, h_next, hp_next, h_f32, B, H, f);
  else if (ksw <= 4)
    launch(lstm_step_kernel<U, 4>, grid, blk, 0, st, gx_t, wp, hp_prev, c, h_next, hp_next, h_f32, B, H, f);
  else if (ksw <= 8)
    launch(lstm_step_kernel<U, 8>, grid, blk, 0, st, gx_t, wp, hp_prev, c, h_next, hp_next, h_f32, B, H, f);
  else
    launch(lstm_step_kernel<U, 16>, grid, blk, 0, st, gx_t, wp, hp_prev, c, h_next, hp_next, h_f32, B, H, f);
}

static dstack_status lstm_check(int B, int H) {
  DS_CHECK(B >= 1 && B <= 32, DSTACK_E_UNSUPPORTED, "lstm: batch must be 1..32");
  // depth is consumed in steps of 32; a block owns 4U hidden units (4U divides 32)
  DS_CHECK(H % 32 == 0 && H >= 32 && H <= 2048, DSTACK_E_UNSUPPORTED, "lstm: H must be a multiple of 32, <= 2048");
  return DSTACK_OK;
}

dstack_status launch_lstm_pack_whh(const bf16* w_hh, bf16* wp, int H, hipStream_t st) {
  dstack_status s = lstm_check(1, H);
  if (s != DSTACK_OK) return s;
  const long vecs = (long)H * H / 2;
  launch(lstm_pack_whh_kernel, dim3((unsigned)((vecs + 255) / 256)), dim3(256), 0, st, w_hh, wp, H);
  DS_HIP(hipGetLastError());
  return DSTACK_OK;
}

dstack_status launch_lstm_step(const float* gx_t, const bf16* wp, const bf16* hp_prev, float* c, bf16* h_next,
                               bf16* hp_next, float* h_f32, int B, int H, bool first, int n_cu, hipStream_t st) {
  dstack_status s = lstm_check(B, H);
  if (s != DSTACK_OK) return s;
  const int nks = H / 32, ksw = (nks + 3) / 4;
  const int u = lstm_units_per_block(B, H, n_cu);
  const dim3 grid(H / (4 * u));
  const int f = first ? 1 : 0;
  if (u == 1)
    launch_lstm_u<1>(ksw, grid, st, gx_t, wp, hp_prev, c, h_next, hp_next, h_f32, B, H, f);
  else if (u == 2)
    launch_lstm_u<2>(ksw, grid, st, gx_t, wp, hp_prev, c, h_next, hp_next, h_f32, B, H, f);
  else
    launch_lstm_u<4>(ksw, grid, st, gx_t, wp, hp_prev, c, h_next, hp_next, h_f32, B, H, f);
  DS_HIP(hipGetLastError());
  return DSTACK_OK;
}

}  // namespace dstack
