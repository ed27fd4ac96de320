// MobileNetV2's expand 1x1 conv + BN + ReLU6 fused with the depthwise 3x3 +
// BN + ReLU6 that consumes it (the inverted residual block of Sec. 3's
// MobileNet).  The expanded tensor E (6x the input channels, the largest
// activation of the block) never leaves the chip: a block takes an output
// tile of TR x TW pixels and a chunk of CB expanded channels, computes E for
// the tile plus its one-pixel halo on the matrix cores into LDS, then runs
// the depthwise filter from LDS and writes only the depthwise output D.
//
// Expand: GEMM rows = the CB expanded channels (weights [Ce][Cin], A
// operand, in registers for the block), columns = the E tile's pixels (B
// operand, 8 consecutive input channels of one pixel per lane, 16-byte loads
// from the NHWC input), depth = Cin in steps of 32 (zero beyond Cin).  The
// result (4 consecutive channels of one pixel per lane) goes through the BN
// scale/shift and ReLU6 to bf16 in LDS, [pixel][channel] with 16 bytes of
// padding per pixel; E pixels outside the image are stored as zeros, which
// is the depthwise filter's zero padding.  Depthwise: one thread per (output
// pixel, 8 channels), 9 16-byte LDS reads, fp32 accumulate.
#include <hip/hip_ext.h>

#include "common.hpp"

namespace dstack {

struct ExpandDwArgs {
  const bf16* x;     // [N][H][W][Cin]
  const bf16* we;    // [Ce][Cin]
  const float* se;   // expand BN scale [Ce]
  const float* he;   // expand BN shift [Ce]
  const bf16* wd;    // [3][3][Ce]
  const float* sd;   // depthwise BN scale [Ce]
  const float* hd;   // depthwise BN shift [Ce]
  bf16* y;           // [N][Ho][Wo][Ce]
  int N, H, W, Cin, Ce, Ho, Wo, stride;
  int act_e, act_d;
  int TR, TW, ER, EC, EM;  // output tile, E tile rows / cols / pixels (EM <= 256)
  int tiles_h, tiles_w, chunks, blocks;
};

constexpr int ED_MAX_EM = 256;

// activation as a clamp to [lo, hi]: none (-inf, inf), ReLU (0, inf), ReLU6 (0, 6)
__device__ __forceinline__ float2 act_bounds(int act) {
  return float2{act == ACT_NONE ? -INFINITY : 0.0f, act == ACT_RELU6 ? 6.0f : INFINITY};
}

template <int CB, int DS>
__global__ __launch_bounds__(256) void expand_dw_kernel(ExpandDwArgs a) {
  constexpr int RB = CB / 16;       // MFMA row blocks of expanded channels
  constexpr int PS = CB * 2 + 16;   // LDS bytes per E pixel (padded)
  constexpr int CV = CB / 8;        // 8-channel vectors per pixel
  constexpr int WROW = DS * 64 + 16;  // LDS bytes per expand-weight row (depth padded to DS*32, + 16 against conflicts)
  __shared__ __attribute__((aligned(16))) unsigned char et[ED_MAX_EM * PS];
  __shared__ __attribute__((aligned(16))) unsigned char wel[CB * WROW];  // expand weights of the chunk
  __shared__ __attribute__((aligned(16))) bf16 wdl[9 * CB];              // depthwise weights of the chunk
  __shared__ __attribute__((aligned(16))) float bnl[4 * CB];             // se, he, sd, hd of the chunk

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, quad = lane >> 4;
  // XCD-aware order: consecutive logical blocks (the channel chunks of one
  // spatial tile, then the next tile) share an XCD and its L2
  int blk;
  {
    const int L = blockIdx.x, q = a.blocks >> 3, r = a.blocks & 7, xcd = L & 7, i = L >> 3;
    blk = xcd * q + min(xcd, r) + i;
  }
  const int chunk = blk % a.chunks;
  int t = blk / a.chunks;
  const int tw = t % a.tiles_w;
  t /= a.tiles_w;
  const int th = t % a.tiles_h;
  const int n = t / a.tiles_h;
  const int c0 = chunk * CB;
  const int ho0 = th * a.TR, wo0 = tw * a.TW;
  const int er0 = ho0 * a.stride - 1, ec0 = wo0 * a.stride - 1;

  // stage the chunk's weights and BN in LDS (each is read by many lanes):
  // expand rows c0.. as 16-byte vectors (zero past Cin), depthwise [9][CB], BN
  {
    const int vpr = DS * 4;  // 16-byte vectors per padded row
    for (int v = tid; v < CB * vpr; v += 256) {
      const int row = v / vpr, col = (v - row * vpr) * 8;
      const uint4 w = col < a.Cin ? *reinterpret_cast<const uint4*>(a.we + (long)(c0 + row) * a.Cin + col) : uint4{};
      *reinterpret_cast<uint4*>(wel + row * WROW + col * 2) = w;
    }
    for (int v = tid; v < 9 * CB / 8; v += 256) {
      const int k = v / (CB / 8), cvv = v - k * (CB / 8);
      *reinterpret_cast<uint4*>(wdl + k * CB + cvv * 8) = *reinterpret_cast<const uint4*>(a.wd + k * a.Ce + c0 + cvv * 8);
    }
    for (int v = tid; v < CB; v += 256) {
      bnl[v] = a.se[c0 + v];
      bnl[CB + v] = a.he[c0 + v];
      bnl[2 * CB + v] = a.sd[c0 + v];
      bnl[3 * CB + v] = a.hd[c0 + v];
    }
  }
  // the E tile's input fragments: wave w takes pixel groups w, w+4, w+8, w+12 (EM <= 256)
  const int groups = (a.EM + 15) / 16;
  bf16x8 b[4][DS];
  bool inside[4];
  int pxs[4];
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int g = wave + 4 * u;
    const int px = g * 16 + (lane & 15);
    const int er = px / a.EC, ec = px - (px / a.EC) * a.EC;
    const int hi = er0 + er, wi = ec0 + ec;
    pxs[u] = px;
    inside[u] = g < groups && px < a.EM && (unsigned)hi < (unsigned)a.H && (unsigned)wi < (unsigned)a.W;
    const bf16* xp = a.x + (((long)n * a.H + (inside[u] ? hi : 0)) * a.W + (inside[u] ? wi : 0)) * a.Cin;
#pragma unroll
    for (int ds = 0; ds < DS; ++ds) {
      const int c = ds * 32 + quad * 8;
      b[u][ds] = inside[u] && c < a.Cin ? *reinterpret_cast<const bf16x8*>(xp + c) : bf16x8{};
    }
  }
  __syncthreads();  // weights and BN staged

  // expand weights: row rb*16 + lane%16 of the chunk, depth ds*32 + quad*8 .. +8
  bf16x8 wa[RB][DS];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int ds = 0; ds < DS; ++ds)
      wa[rb][ds] = *reinterpret_cast<const bf16x8*>(wel + (rb * 16 + (lane & 15)) * WROW + (ds * 32 + quad * 8) * 2);
  // expand BN for this lane's channels rb*16 + 4*quad + i
  f32x4 sce[RB], she[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    sce[rb] = *reinterpret_cast<const f32x4*>(bnl + rb * 16 + 4 * quad);
    she[rb] = *reinterpret_cast<const f32x4*>(bnl + CB + rb * 16 + 4 * quad);
  }
  const float2 be = act_bounds(a.act_e), bd = act_bounds(a.act_d);

  // ---- expand on the matrix cores, BN + activation, bf16 E tile in LDS ----
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    if (wave + 4 * u >= groups) break;  // wave-uniform
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      f32x4 acc = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa[rb][ds], b[u][ds], acc, 0, 0, 0);
      bf16x4 e;
#pragma unroll
      for (int i = 0; i < 4; ++i)
        e[i] = (bf16)(inside[u] ? fminf(fmaxf(acc[i] * sce[rb][i] + she[rb][i], be.x), be.y) : 0.0f);
      if (pxs[u] < a.EM) *reinterpret_cast<bf16x4*>(et + pxs[u] * PS + (rb * 16 + 4 * quad) * 2) = e;
    }
  }
  __syncthreads();
  // ---- depthwise 3x3 from the E tile: thread = fixed 8-channel vector cv,
  // pixels tid / CV, + PT, ...; its 9 weight vectors and BN in registers ----
  constexpr int PT = 256 / CV;  // pixels in flight per pass
  if (tid >= PT * CV) return;
  const int cv = tid % CV;
  const int ch = c0 + cv * 8;
  bf16x8 wv[9];
#pragma unroll
  for (int k = 0; k < 9; ++k) wv[k] = *reinterpret_cast<const bf16x8*>(wdl + k * CB + cv * 8);
  const f32x4 s0 = *reinterpret_cast<const f32x4*>(bnl + 2 * CB + cv * 8);
  const f32x4 s1 = *reinterpret_cast<const f32x4*>(bnl + 2 * CB + cv * 8 + 4);
  const f32x4 h0 = *reinterpret_cast<const f32x4*>(bnl + 3 * CB + cv * 8);
  const f32x4 h1 = *reinterpret_cast<const f32x4*>(bnl + 3 * CB + cv * 8 + 4);

  const int npix = a.TR * a.TW;
  for (int pix = tid / CV; pix < npix; pix += PT) {
    const int r = pix / a.TW, c = pix - (pix / a.TW) * a.TW;
    const int ho = ho0 + r, wo = wo0 + c;
    if (ho >= a.Ho || wo >= a.Wo) continue;
    float acc[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) acc[j] = 0.f;
#pragma unroll
    for (int kr = 0; kr < 3; ++kr)
#pragma unroll
      for (int kc = 0; kc < 3; ++kc) {
        const int e = (r * a.stride + kr) * a.EC + c * a.stride + kc;
        const bf16x8 v = *reinterpret_cast<const bf16x8*>(et + e * PS + cv * 16);
#pragma unroll
        for (int j = 0; j < 8; ++j) acc[j] += (float)v[j] * (float)wv[kr * 3 + kc][j];
      }
    bf16x8 o;
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      o[j] = (bf16)fminf(fmaxf(acc[j] * s0[j] + h0[j], bd.x), bd.y);
      o[j + 4] = (bf16)fminf(fmaxf(acc[j + 4] * s1[j] + h1[j], bd.x), bd.y);
    }
    *reinterpret_cast<bf16x8*>(a.y + (((long)n * a.Ho + ho) * a.Wo + wo) * a.Ce + ch) = o;
  }
}

// Output tile TR x TW with the most outputs whose E tile (plus halo) has at
// most ED_MAX_EM pixels; ties to the wider tile.
static void expand_dw_tile(int Ho, int Wo, int stride, int* TR, int* TW) {
  int best = 0;
  *TR = *TW = 1;
  for (int tr = 1; tr <= Ho; ++tr)
    for (int tw = 1; tw <= Wo; ++tw) {
      const int em = ((tr - 1) * stride + 3) * ((tw - 1) * stride + 3);
      if (em > ED_MAX_EM) break;
      // count the outputs of all tiles, penalising the partial ones at the edges
      const long tiles = (long)((Ho + tr - 1) / tr) * ((Wo + tw - 1) / tw);
      const int useful = (int)((long)Ho * Wo * 1000 / (tiles * tr * tw));  // permille of computed outputs kept
      const int score = tr * tw * useful;
      if (score > best || (score == best && tw > *TW)) {
        best = score;
        *TR = tr;
        *TW = tw;
      }
    }
}

template <int CB>
static void expand_dw_launch_cb(const ExpandDwArgs& a, int ds, hipStream_t st) {
  const dim3 grid((unsigned)a.blocks);
  switch (ds) {
    case 1: hipLaunchKernelGGL((expand_dw_kernel<CB, 1>), grid, dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL((expand_dw_kernel<CB, 2>), grid, dim3(256), 0, st, a); break;
    case 3: hipLaunchKernelGGL((expand_dw_kernel<CB, 3>), grid, dim3(256), 0, st, a); break;
    case 4: hipLaunchKernelGGL((expand_dw_kernel<CB, 4>), grid, dim3(256), 0, st, a); break;
    default: hipLaunchKernelGGL((expand_dw_kernel<CB, 5>), grid, dim3(256), 0, st, a); break;
  }
}

dstack_status launch_expand_dw(const bf16* x, int N, int H, int W, int Cin, const bf16* we, int Ce, const float* se,
                               const float* he, int act_e, const bf16* wd, int stride, const float* sd,
                               const float* hd, int act_d, bf16* y, hipStream_t st) {
  DS_CHECK(x && we && se && he && wd && sd && hd && y, DSTACK_E_INVALID, "expand_dw: null pointer");
  DS_CHECK(N > 0 && H > 0 && W > 0 && (stride == 1 || stride == 2), DSTACK_E_INVALID, "expand_dw: bad shape");
  DS_CHECK(Cin % 8 == 0 && Cin <= 160, DSTACK_E_UNSUPPORTED, "expand_dw: Cin must be a multiple of 8, at most 160");
  DS_CHECK(Ce % 48 == 0 || Ce % 64 == 0, DSTACK_E_UNSUPPORTED, "expand_dw: Ce must be a multiple of 48 or 64");
  DS_CHECK(act_e >= 0 && act_e <= 2 && act_d >= 0 && act_d <= 2, DSTACK_E_INVALID, "expand_dw: act must be 0, 1 or 2");
  ExpandDwArgs a;
  a.x = x; a.we = we; a.se = se; a.he = he; a.wd = wd; a.sd = sd; a.hd = hd; a.y = y;
  a.N = N; a.H = H; a.W = W; a.Cin = Cin; a.Ce = Ce; a.stride = stride; a.act_e = act_e; a.act_d = act_d;
  a.Ho = out_dim(H, 3, stride, 1);
  a.Wo = out_dim(W, 3, stride, 1);
  DS_CHECK((long)N * H * W * Cin < (1L << 31) && (long)N * a.Ho * a.Wo * Ce < (1L << 31), DSTACK_E_UNSUPPORTED,
           "expand_dw: tensor too large");
  expand_dw_tile(a.Ho, a.Wo, stride, &a.TR, &a.TW);
  a.ER = (a.TR - 1) * stride + 3;
  a.EC = (a.TW - 1) * stride + 3;
  a.EM = a.ER * a.EC;
  a.tiles_h = ceil_div(a.Ho, a.TR);
  a.tiles_w = ceil_div(a.Wo, a.TW);
  // 64-channel chunks (each pixel's chunk of the output one whole 128-byte
  // line) where they divide Ce and still leave 384 or more blocks; else 48
  const long tiles = (long)N * a.tiles_h * a.tiles_w;
  const int cb = (Ce % 64 == 0 && (Ce % 48 != 0 || tiles * (Ce / 64) >= 384)) ? 64 : 48;
  a.chunks = Ce / cb;
  const long blocks = tiles * a.chunks;
  DS_CHECK(blocks < (1L << 31), DSTACK_E_UNSUPPORTED, "expand_dw: grid too large");
  a.blocks = (int)blocks;
  if (cb == 64)
    expand_dw_launch_cb<64>(a, ceil_div(Cin, 32), st);
  else
    expand_dw_launch_cb<48>(a, ceil_div(Cin, 32), st);
  DS_HIP(hipGetLastError());
  return DSTACK_OK;
}

}  // namespace dstack
