// Implicit-GEMM convolution on gfx950 matrix cores (bf16 in, fp32 accumulate).
//
// The convolution is the compute-bound layer class of the paper's
// arithmetic-intensity table (Sec. 4.1): y = act(scale * conv(x, w) + shift
// [+ res]) with NHWC activations and KRSC weights.  As a GEMM:
//   rows    = output channels k        (K, "BN" tile)
//   columns = output pixels (n,ho,wo)  (M = N*Ho*Wo, "BM" tile)
//   depth   = (r, s, c)                (Kg = R*S*C, contiguous in both operands)
// The weight row for channel k is contiguous over (r,s,c); the im2col row of
// a pixel is gathered on the fly, 8 channels (16 bytes) at a time, which
// needs C % 8 == 0 (3-channel stems are zero-padded to 8 before the call).
//
// Block: 256 threads = 4 waves in a 2x2 grid over the (BN x BM) tile; each
// wave owns (BN/2 x BM/2) and issues v_mfma_f32_16x16x32_bf16 on it.  Tiles
// of BK = 64 depth are staged global -> registers -> LDS with a two-stage
// LDS ring, so the next tile's global loads are in flight during the current
// tile's MFMAs.  Operand layouts of the 16x16x32 bf16 MFMA (checked on the
// device): lane l holds A[l%16][8*(l/16) .. +8) and B[8*(l/16) .. +8)[l%16];
// the result holds C[4*(l/16)+i][l%16], i = 0..3, so each lane ends with 4
// consecutive output channels of one pixel: one 8-byte bf16 store.
//
// Split-K: with gridDim.z = splits > 1 each z-slice accumulates a range of
// depth tiles and writes raw fp32 partial sums to a workspace; a second
// kernel sums the slices and applies the epilogue.
#include "common.hpp"

namespace dstack {

struct ConvArgs {
  const bf16* x;
  const bf16* w;
  const float* scale;  // nullptr: 1
  const float* shift;  // nullptr: 0
  const bf16* res;     // nullptr: no residual
  void* y;
  float* partial;      // split-K workspace [splits][M][K]
  int N, H, W, C, K, R, S, stride, pad, Ho, Wo;
  int M, Kg;
  int act;
  int kt_per_split;
};

constexpr int BK = 64;
constexpr int LDK = BK + 8;   // LDS row pitch (bf16): 144 B, spreads 16 rows over all banks
constexpr int CPR = BK / 8;   // 16-byte chunks per tile row
constexpr int RSTEP = 256 / CPR;

__device__ __forceinline__ void store_out4(void* y, bool f32, long idx, const float v[4]) {
  if (f32) {
    f32x4 o = {v[0], v[1], v[2], v[3]};
    *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(y) + idx) = o;
  } else {
    bf16x4 o = {(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3]};
    *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(y) + idx) = o;
  }
}

__device__ __forceinline__ void epilogue4(const ConvArgs& a, bool f32, int px, int ch0, const float acc[4]) {
  float v[4];
  f32x4 sc = a.scale ? *reinterpret_cast<const f32x4*>(a.scale + ch0) : f32x4{1.f, 1.f, 1.f, 1.f};
  f32x4 sh = a.shift ? *reinterpret_cast<const f32x4*>(a.shift + ch0) : f32x4{0.f, 0.f, 0.f, 0.f};
  long idx = (long)px * a.K + ch0;
  bf16x4 r4 = {};
  if (a.res) r4 = *reinterpret_cast<const bf16x4*>(a.res + idx);
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    float t = acc[i] * sc[i] + sh[i];
    if (a.res) t += (float)r4[i];
    v[i] = apply_act(t, a.act);
  }
  store_out4(a.y, f32, idx, v);
}

template <int BN, int BM, bool OUT_F32, bool SPLIT>
__global__ __launch_bounds__(256) void conv_igemm_kernel(ConvArgs a) {
  constexpr int NW = BN * CPR / 256;  // weight chunks per thread
  constexpr int NX = BM * CPR / 256;  // activation chunks per thread
  constexpr int TN = BN / 32;         // 16-row MFMA tiles per wave (channels)
  constexpr int TM = BM / 32;         // 16-col MFMA tiles per wave (pixels)
  static_assert(NW >= 1 && NX >= 1, "tile too small for 256 threads");

  __shared__ __attribute__((aligned(16))) bf16 lds[2][(BN + BM) * LDK];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wn = wave & 1, wm = wave >> 1;
  const int n0 = blockIdx.y * BN;  // first output channel of the tile
  const int m0 = blockIdx.x * BM;  // first output pixel of the tile
  const int kc = tid % CPR;

  // per-row im2col bookkeeping for this thread's activation chunks
  int xbase[NX], hi0[NX], wi0[NX];
  bool xvalid[NX];
#pragma unroll
  for (int i = 0; i < NX; ++i) {
    int m = m0 + tid / CPR + RSTEP * i;
    xvalid[i] = m < a.M;
    int mm = xvalid[i] ? m : 0;
    int wo = mm % a.Wo;
    int t = mm / a.Wo;
    int ho = t % a.Ho;
    int n = t / a.Ho;
    xbase[i] = n * a.H * a.W * a.C;
    hi0[i] = ho * a.stride - a.pad;
    wi0[i] = wo * a.stride - a.pad;
  }

  const int nkt_total = (a.Kg + BK - 1) / BK;
  int kt0 = 0, kt1 = nkt_total;
  if (SPLIT) {
    kt0 = blockIdx.z * a.kt_per_split;
    kt1 = min(nkt_total, kt0 + a.kt_per_split);
  }

  bf16x8 wr[NW], xr[NX];
  const bf16x8 zero8 = {};

  auto load_tiles = [&](int kt) {
    const int k = kt * BK + kc * 8;
    const bool kin = k < a.Kg;
#pragma unroll
    for (int i = 0; i < NW; ++i) {
      int n = n0 + tid / CPR + RSTEP * i;
      wr[i] = (kin && n < a.K) ? *reinterpret_cast<const bf16x8*>(a.w + (long)n * a.Kg + k) : zero8;
    }
    int rs = kin ? k / a.C : 0;
    int c = k - rs * a.C;
    int r = rs / a.S;
    int s = rs - r * a.S;
#pragma unroll
    for (int i = 0; i < NX; ++i) {
      int hi = hi0[i] + r, wi = wi0[i] + s;
      bool ok = kin && xvalid[i] && (unsigned)hi < (unsigned)a.H && (unsigned)wi < (unsigned)a.W;
      xr[i] = ok ? *reinterpret_cast<const bf16x8*>(a.x + xbase[i] + (hi * a.W + wi) * a.C + c) : zero8;
    }
  };
  auto store_tiles = [&](int buf) {
#pragma unroll
    for (int i = 0; i < NW; ++i)
      *reinterpret_cast<bf16x8*>(&lds[buf][(tid / CPR + RSTEP * i) * LDK + kc * 8]) = wr[i];
#pragma unroll
    for (int i = 0; i < NX; ++i)
      *reinterpret_cast<bf16x8*>(&lds[buf][(BN + tid / CPR + RSTEP * i) * LDK + kc * 8]) = xr[i];
  };

  f32x4 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  if (kt0 < kt1) {
    load_tiles(kt0);
    store_tiles(0);
  }
  __syncthreads();

  const int arow = wn * (BN / 2) + (lane & 15);
  const int brow = BN + wm * (BM / 2) + (lane & 15);
  const int koff = (lane >> 4) * 8;

  for (int kt = kt0; kt < kt1; ++kt) {
    const int buf = (kt - kt0) & 1;
    const bool more = kt + 1 < kt1;
    if (more) load_tiles(kt + 1);
#pragma unroll
    for (int ks = 0; ks < BK; ks += 32) {
      bf16x8 af[TN], bfr[TM];
#pragma unroll
      for (int i = 0; i < TN; ++i)
        af[i] = *reinterpret_cast<const bf16x8*>(&lds[buf][(arow + i * 16) * LDK + ks + koff]);
#pragma unroll
      for (int j = 0; j < TM; ++j)
        bfr[j] = *reinterpret_cast<const bf16x8*>(&lds[buf][(brow + j * 16) * LDK + ks + koff]);
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
    if (more) store_tiles(buf ^ 1);
    __syncthreads();
  }

  // epilogue: lane holds channels ch0..ch0+3 of pixel px for each (i, j) tile
#pragma unroll
  for (int i = 0; i < TN; ++i) {
    const int ch0 = n0 + wn * (BN / 2) + i * 16 + (lane >> 4) * 4;
#pragma unroll
    for (int j = 0; j < TM; ++j) {
      const int px = m0 + wm * (BM / 2) + j * 16 + (lane & 15);
      if (px >= a.M || ch0 >= a.K) continue;
      float v[4] = {acc[i][j][0], acc[i][j][1], acc[i][j][2], acc[i][j][3]};
      if (SPLIT) {
        float* p = a.partial + ((long)blockIdx.z * a.M + px) * a.K + ch0;
        *reinterpret_cast<f32x4*>(p) = f32x4{v[0], v[1], v[2], v[3]};
      } else {
        epilogue4(a, OUT_F32, px, ch0, v);
      }
    }
  }
}

// Sum split-K partial slices and apply the epilogue; one thread per 4 channels.
__global__ void splitk_reduce_kernel(ConvArgs a, int splits, int out_f32) {
  long q = (long)blockIdx.x * blockDim.x + threadIdx.x;
  long nq = (long)a.M * (a.K / 4);
  if (q >= nq) return;
  int px = (int)(q / (a.K / 4));
  int ch0 = (int)(q % (a.K / 4)) * 4;
  float v[4] = {0.f, 0.f, 0.f, 0.f};
  for (int s = 0; s < splits; ++s) {
    f32x4 p = *reinterpret_cast<const f32x4*>(a.partial + ((long)s * a.M + px) * a.K + ch0);
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] += p[i];
  }
  epilogue4(a, out_f32 != 0, px, ch0, v);
}

template <int BN, int BM>
static void launch_cfg(const ConvArgs& a, bool f32, int splits, hipStream_t st) {
  dim3 grid(ceil_div(a.M, BM), ceil_div(a.K, BN), splits);
  if (splits > 1)
    hipLaunchKernelGGL((conv_igemm_kernel<BN, BM, false, true>), grid, dim3(256), 0, st, a);
  else if (f32)
    hipLaunchKernelGGL((conv_igemm_kernel<BN, BM, true, false>), grid, dim3(256), 0, st, a);
  else
    hipLaunchKernelGGL((conv_igemm_kernel<BN, BM, false, false>), grid, dim3(256), 0, st, a);
}

// Split-K workspace: a grow-only device buffer per stream would be needed for
// concurrent splits; the caller passes it through ConvArgs.partial instead.
struct ConvPlan {
  int bn, bm, splits;
};

// Tile and split choice from the GEMM shape and the CUs of the partition.
static ConvPlan choose_plan(int M, int K, int Kg, int n_cu) {
  ConvPlan p;
  p.bn = K >= 128 ? 128 : (K >= 64 ? 64 : 32);
  p.bm = (p.bn == 32) ? 256 : 128;
  long tiles = (long)ceil_div(M, p.bm) * ceil_div(K, p.bn);
  if (tiles < n_cu && p.bn == 128 && M <= 64 * n_cu) {
    p.bm = 64;
    tiles = (long)ceil_div(M, p.bm) * ceil_div(K, p.bn);
  }
  p.splits = 1;
  int nkt = ceil_div(Kg, BK);
  // too few tiles to cover the partition and a deep reduction: split the depth
  while (tiles * p.splits * 2 <= n_cu && nkt / (p.splits * 2) >= 4 && p.splits < 16) p.splits *= 2;
  return p;
}

size_t conv_splitk_workspace_bytes(int M, int K, int Kg, int n_cu) {
  ConvPlan p = choose_plan(M, K, Kg, n_cu);
  return p.splits > 1 ? (size_t)p.splits * M * K * sizeof(float) : 0;
}

dstack_status launch_conv2d_ws(const bf16* x, int N, int H, int W, int C, const bf16* w, int K, int R, int S,
                               int stride, int pad, const float* scale, const float* shift, const bf16* res,
                               int act, void* y, bool out_fp32, int n_cu, float* splitk_ws, size_t splitk_bytes,
                               hipStream_t st) {
  DS_CHECK(C % 8 == 0, DSTACK_E_UNSUPPORTED, "conv2d: C must be a multiple of 8");
  DS_CHECK(K % 4 == 0, DSTACK_E_UNSUPPORTED, "conv2d: K must be a multiple of 4");
  DS_CHECK(N > 0 && H > 0 && W > 0 && K > 0 && R > 0 && S > 0 && stride > 0 && pad >= 0, DSTACK_E_INVALID,
           "conv2d: bad shape");
  ConvArgs a;
  a.x = x; a.w = w; a.scale = scale; a.shift = shift; a.res = res; a.y = y; a.partial = nullptr;
  a.N = N; a.H = H; a.W = W; a.C = C; a.K = K; a.R = R; a.S = S; a.stride = stride; a.pad = pad;
  a.Ho = out_dim(H, R, stride, pad);
  a.Wo = out_dim(W, S, stride, pad);
  DS_CHECK(a.Ho > 0 && a.Wo > 0, DSTACK_E_INVALID, "conv2d: empty output");
  DS_CHECK((long)N * H * W * C < (1L << 31) && (long)N * a.Ho * a.Wo * K < (1L << 31) && (long)K * R * S * C < (1L << 31),
           DSTACK_E_UNSUPPORTED, "conv2d: tensor too large for 32-bit indexing");
  a.M = N * a.Ho * a.Wo;
  a.Kg = R * S * C;
  a.act = act;
  ConvPlan p = choose_plan(a.M, K, a.Kg, n_cu);
  if (p.splits > 1 && (splitk_ws == nullptr || splitk_bytes < (size_t)p.splits * a.M * K * sizeof(float)))
    p.splits = 1;
  int nkt = ceil_div(a.Kg, BK);
  a.kt_per_split = ceil_div(nkt, p.splits);
  p.splits = ceil_div(nkt, a.kt_per_split);  // no empty slices
  if (p.splits > 1) a.partial = splitk_ws;
#define DS_CONV_CASE(BN_, BM_) \
  if (p.bn == BN_ && p.bm == BM_) launch_cfg<BN_, BM_>(a, out_fp32, p.splits, st);
  DS_CONV_CASE(128, 128)
  else DS_CONV_CASE(128, 64)
  else DS_CONV_CASE(64, 128)
  else DS_CONV_CASE(32, 256)
#undef DS_CONV_CASE
  if (p.splits > 1) {
    long nq = (long)a.M * (K / 4);
    hipLaunchKernelGGL(splitk_reduce_kernel, dim3((unsigned)((nq + 255) / 256)), dim3(256), 0, st, a, p.splits,
                       out_fp32 ? 1 : 0);
  }
  DS_HIP(hipGetLastError());
  return DSTACK_OK;
}

dstack_status launch_conv2d(const bf16* x, int N, int H, int W, int C, const bf16* w, int K, int R, int S,
                            int stride, int pad, const float* scale, const float* shift, const bf16* res, int act,
                            void* y, bool out_fp32, int n_cu, hipStream_t st) {
  return launch_conv2d_ws(x, N, H, W, C, w, K, R, S, stride, pad, scale, shift, res, act, y, out_fp32, n_cu,
                          nullptr, 0, st);
}

}  // namespace dstack
