// MobileNetV2's expand 1x1 conv + BN + ReLU6 fused with the depthwise 3x3 +
// BN + ReLU6 that consumes it (the inverted residual block of Sec. 3's
// MobileNet).  The expanded tensor E (6x the input channels, the largest
// activation of the block) never leaves the chip: a block takes an output
// tile of TR x TW pixels and a chunk of CB expanded channels, computes E for
// the tile plus its one-pixel halo on the matrix cores into LDS, then runs
// the depthwise filter from LDS and writes only the depthwise output D.
//
// E tile: ER rows x ECP columns (the halo'd width EC rounded up to even),
// pixels numbered row-major.  In LDS it is stored as column pairs: word
// (pair, c) holds channel c of the even and the odd column of one pair as
// two bf16, CB + 8 words per pair (the 8 spread the four quads of a wave
// over distinct banks).
//
// Expand: GEMM rows = 16 E pixels (A operand, 8 consecutive input channels
// of one pixel per lane, 16-byte loads from the NHWC input), columns = 16
// expanded channels (B operand, weights [Ce][Cin] staged in LDS), depth =
// Cin in steps of 32 (zero beyond Cin).  A lane's result is one channel of
// 4 consecutive pixels, i.e. two column pairs, which go through BN and the
// activation to two LDS words; E pixels outside the image are stored as
// zeros, which is the depthwise filter's zero padding.
//
// Depthwise: a thread takes 4 channels of one output pixel (stride 2) or of
// two horizontally adjacent ones (stride 1).  Per filter row it reads the
// column pairs under the window (16 bytes each) and accumulates with
// bf16 dot products of two taps: at stride 1 the even output takes taps
// (0,1) from the first pair and tap 2 from the next pair's even column, the
// odd output tap 0 from the first pair's odd column and taps (1,2) from the
// next pair, the unused half weighted by zero; fp32 accumulate.
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
  int TR, TW, ER, EC, ECP, EM;  // output tile; E tile rows, cols, cols rounded up to even, pixels ER*ECP (<= 256)
  int tiles_h, tiles_w, chunks, blocks;
  FastDiv div_chunks, div_tw, div_th, div_ecp, div_twi;  // by chunks, tiles_w, tiles_h, ECP, work items per tile row
};

constexpr int ED_MAX_EM = 256;

// activation as a clamp to [lo, hi]: none (-inf, inf), ReLU (0, inf), ReLU6 (0, 6)
__device__ __forceinline__ float2 act_bounds(int act) {
  return float2{act == ACT_NONE ? -INFINITY : 0.0f, act == ACT_RELU6 ? 6.0f : INFINITY};
}

typedef __attribute__((__vector_size__(2 * sizeof(__bf16)))) __bf16 bf16x2;

__device__ __forceinline__ float dot2(unsigned e, bf16x2 w, float acc) {
  return __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, e), w, acc, false);
}

typedef float f32x2 __attribute__((ext_vector_type(2)));

// two floats to round-to-nearest-even bf16 in one packed conversion
__device__ __forceinline__ unsigned pack_bf16x2(float lo, float hi) {
  return __builtin_bit_cast(unsigned, __builtin_convertvector((f32x2{lo, hi}), bf16x2));
}

template <int CB, int DS, int S>
__global__ __launch_bounds__(256) void expand_dw_kernel(ExpandDwArgs a) {
  constexpr int RB = CB / 16;       // MFMA column blocks of expanded channels
  constexpr int PW = CB + 8;        // LDS words per E column pair
  constexpr int CG = CB / 4;        // 4-channel groups of the depthwise phase
  constexpr int WROW = DS * 64 + 16;  // LDS bytes per expand-weight row (depth padded to DS*32, + 16 against conflicts)
  __shared__ __attribute__((aligned(16))) unsigned et[ED_MAX_EM / 2 * PW];
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
  int t = a.div_chunks.div(blk);
  const int chunk = blk - t * a.chunks;
  int t2 = a.div_tw.div(t);
  const int tw = t - t2 * a.tiles_w;
  const int n = a.div_th.div(t2);
  const int th = t2 - n * a.tiles_h;
  const int c0 = chunk * CB;
  const int ho0 = th * a.TR, wo0 = tw * a.TW;
  const int er0 = ho0 * S - 1, ec0 = wo0 * S - 1;

  // Every global load of the prologue is issued before the first LDS store,
  // so the block waits for one memory round trip rather than one per array:
  // the chunk's expand rows c0.. as 16-byte vectors (zero past Cin), its
  // depthwise weights [9][CB] and its four BN vectors (each read by many
  // lanes, so staged in LDS), then the E tile's input fragments (registers).
  // Element offsets are 32-bit (the host bounds every tensor below 2^31).
  constexpr int VPR = DS * 4;                 // 16-byte vectors per padded expand row
  constexpr int WV = (CB * VPR + 255) / 256;  // expand-weight vectors per thread
  uint4 wst[WV];
#pragma unroll
  for (int i = 0; i < WV; ++i) {
    const int v = tid + i * 256, row = v / VPR, col = (v - row * VPR) * 8;
    wst[i] = v < CB * VPR && col < a.Cin ? *reinterpret_cast<const uint4*>(a.we + ((c0 + row) * a.Cin + col))
                                          : uint4{};
  }
  static_assert(9 * CB / 8 <= 256 && 4 * CB <= 256, "one depthwise vector and one BN value per thread");
  const int dk = tid / (CB / 8), dcv = tid - dk * (CB / 8);
  const uint4 dst = tid < 9 * CB / 8 ? *reinterpret_cast<const uint4*>(a.wd + (dk * a.Ce + c0 + dcv * 8)) : uint4{};
  const int bk = tid / CB, bc = tid - bk * CB;
  const float* bsrc = bk == 0 ? a.se : bk == 1 ? a.he : bk == 2 ? a.sd : a.hd;
  const float bst = tid < 4 * CB ? bsrc[c0 + bc] : 0.0f;
  // the E tile's input fragments: wave w takes pixel groups w, w+4, w+8, w+12 (EM <= 256)
  const int groups = (a.EM + 15) / 16;
  bf16x8 b[4][DS];
  bool inside[4];
  const int xn = n * a.H;
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int g = wave + 4 * u;
    const int px = g * 16 + (lane & 15);
    const int er = a.div_ecp.div(px), ec = px - er * a.ECP;
    const int hi = er0 + er, wi = ec0 + ec;
    inside[u] = g < groups && px < a.EM && (unsigned)hi < (unsigned)a.H && (unsigned)wi < (unsigned)a.W;
    const bf16* xp = a.x + (((xn + (inside[u] ? hi : 0)) * a.W + (inside[u] ? wi : 0)) * a.Cin + quad * 8);
#pragma unroll
    for (int ds = 0; ds < DS; ++ds)
      b[u][ds] = inside[u] && ds * 32 + quad * 8 < a.Cin ? *reinterpret_cast<const bf16x8*>(xp + ds * 32) : bf16x8{};
  }
#pragma unroll
  for (int i = 0; i < WV; ++i) {
    const int v = tid + i * 256, row = v / VPR, col = (v - row * VPR) * 8;
    if (v < CB * VPR) *reinterpret_cast<uint4*>(wel + row * WROW + col * 2) = wst[i];
  }
  if (tid < 9 * CB / 8) *reinterpret_cast<uint4*>(wdl + dk * CB + dcv * 8) = dst;
  if (tid < 4 * CB) bnl[tid] = bst;
  __syncthreads();  // weights and BN staged

  // expand weights: channel rb*16 + lane%16 of the chunk, depth ds*32 + quad*8 .. +8
  bf16x8 wa[RB][DS];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb)
#pragma unroll
    for (int ds = 0; ds < DS; ++ds)
      wa[rb][ds] = *reinterpret_cast<const bf16x8*>(wel + (rb * 16 + (lane & 15)) * WROW + (ds * 32 + quad * 8) * 2);
  float sce[RB], she[RB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    sce[rb] = bnl[rb * 16 + (lane & 15)];
    she[rb] = bnl[CB + rb * 16 + (lane & 15)];
  }
  const float2 be = act_bounds(a.act_e), bd = act_bounds(a.act_d);

  // ---- expand on the matrix cores, BN + activation, bf16 column pairs in LDS ----
#pragma unroll
  for (int u = 0; u < 4; ++u) {
    const int g = wave + 4 * u;
    if (g >= groups) break;  // wave-uniform
    f32x4 acc[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      acc[rb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int ds = 0; ds < DS; ++ds) acc[rb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(b[u][ds], wa[rb][ds], acc[rb], 0, 0, 0);
    }
    unsigned* dstp = et + (g * 8 + 2 * quad) * PW + (lane & 15);
    // lane p of the first quad loaded pixel g*16 + p; this lane's results are
    // pixels g*16 + 4*quad + i
    const unsigned long long inmask = __ballot(inside[u]);
    if (inmask == ~0ull) {  // the whole group lies in the image (wave-uniform)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        float v[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) v[i] = __builtin_amdgcn_fmed3f(acc[rb][i] * sce[rb] + she[rb], be.x, be.y);
        dstp[rb * 16] = pack_bf16x2(v[0], v[1]);
        dstp[rb * 16 + PW] = pack_bf16x2(v[2], v[3]);
      }
    } else {  // E outside the image is the depthwise filter's zero padding
      const unsigned live = (unsigned)(inmask >> (4 * quad)) & 15u;
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) {
        float v[4];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
          const float e = __builtin_amdgcn_fmed3f(acc[rb][i] * sce[rb] + she[rb], be.x, be.y);
          v[i] = (live >> i) & 1u ? e : 0.0f;
        }
        dstp[rb * 16] = pack_bf16x2(v[0], v[1]);
        dstp[rb * 16 + PW] = pack_bf16x2(v[2], v[3]);
      }
    }
  }
  __syncthreads();

  // ---- depthwise 3x3 from the E tile: thread = fixed 4-channel group cg,
  // work items tid / CG, + PT, ...; its tap-pair weights and BN in registers ----
  constexpr int PT = 256 / CG;  // work items in flight per pass
  if (tid >= PT * CG) return;
  const int cg = tid % CG;
  bf16x2 w01[3][4], w2z[3][4];  // (tap 0, tap 1) and (tap 2, 0) of each filter row
  bf16x2 wz0[3][4], w12[3][4];  // (0, tap 0) and (tap 1, tap 2), stride 1 only
  const bf16 zero = (bf16)0.0f;
#pragma unroll
  for (int kr = 0; kr < 3; ++kr) {
    const bf16x4 t0 = *reinterpret_cast<const bf16x4*>(wdl + (kr * 3 + 0) * CB + cg * 4);
    const bf16x4 t1 = *reinterpret_cast<const bf16x4*>(wdl + (kr * 3 + 1) * CB + cg * 4);
    const bf16x4 t2 = *reinterpret_cast<const bf16x4*>(wdl + (kr * 3 + 2) * CB + cg * 4);
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      w01[kr][j] = bf16x2{t0[j], t1[j]};
      w2z[kr][j] = bf16x2{t2[j], zero};
      wz0[kr][j] = bf16x2{zero, t0[j]};
      w12[kr][j] = bf16x2{t1[j], t2[j]};
    }
  }
  const f32x4 sd = *reinterpret_cast<const f32x4*>(bnl + 2 * CB + cg * 4);
  const f32x4 hd = *reinterpret_cast<const f32x4*>(bnl + 3 * CB + cg * 4);
  bf16* const ybase = a.y + (c0 + cg * 4);
  auto store = [&](const float* acc, int ho, int wo) {
    float o[4];
#pragma unroll
    for (int j = 0; j < 4; ++j) o[j] = __builtin_amdgcn_fmed3f(acc[j] * sd[j] + hd[j], bd.x, bd.y);
    *reinterpret_cast<uint2*>(ybase + ((n * a.Ho + ho) * a.Wo + wo) * a.Ce) =
        uint2{pack_bf16x2(o[0], o[1]), pack_bf16x2(o[2], o[3])};
  };
  const int ECP2 = a.ECP / 2;  // column pairs per E row
  // work item (row r, column c of the tile; output column pairs at stride
  // 1), stepped by PT items per pass without dividing
  const int TWI = S == 1 ? (a.TW + 1) >> 1 : a.TW;
  const int nitems = a.TR * TWI;
  int it = tid / CG;
  int r = a.div_twi.div(it), c = it - r * TWI;
  const int dr = a.div_twi.div(PT), dc = PT - dr * TWI;
  for (; it < nitems; it += PT) {
    const int ho = ho0 + r, wo = wo0 + (S == 1 ? 2 * c : c);
    if (ho < a.Ho && wo < a.Wo) {
      const unsigned* q = et + ((S * r) * ECP2 + c) * PW + cg * 4;
      if (S == 1) {
        float ae[4] = {0.f, 0.f, 0.f, 0.f}, ao[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kr = 0; kr < 3; ++kr) {
          const uint4 p0 = *reinterpret_cast<const uint4*>(q + kr * ECP2 * PW);
          const uint4 p1 = *reinterpret_cast<const uint4*>(q + kr * ECP2 * PW + PW);
          const unsigned e0[4] = {p0.x, p0.y, p0.z, p0.w}, e1[4] = {p1.x, p1.y, p1.z, p1.w};
#pragma unroll
          for (int j = 0; j < 4; ++j) {
            ae[j] = dot2(e1[j], w2z[kr][j], dot2(e0[j], w01[kr][j], ae[j]));
            ao[j] = dot2(e1[j], w12[kr][j], dot2(e0[j], wz0[kr][j], ao[j]));
          }
        }
        store(ae, ho, wo);
        if (2 * c + 1 < a.TW && wo + 1 < a.Wo) store(ao, ho, wo + 1);
      } else {
        float acc[4] = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int kr = 0; kr < 3; ++kr) {
          const uint4 p0 = *reinterpret_cast<const uint4*>(q + kr * ECP2 * PW);
          const uint4 p1 = *reinterpret_cast<const uint4*>(q + kr * ECP2 * PW + PW);
          const unsigned e0[4] = {p0.x, p0.y, p0.z, p0.w}, e1[4] = {p1.x, p1.y, p1.z, p1.w};
#pragma unroll
          for (int j = 0; j < 4; ++j) acc[j] = dot2(e1[j], w2z[kr][j], dot2(e0[j], w01[kr][j], acc[j]));
        }
        store(acc, ho, wo);
      }
    }
    r += dr;
    c += dc;
    if (c >= TWI) {
      c -= TWI;
      ++r;
    }
  }
}

// Output tile TR x TW with the most outputs whose E tile (plus halo, width
// rounded up to even) has at most ED_MAX_EM pixels; ties to the wider tile.
static void expand_dw_tile(int Ho, int Wo, int stride, int* TR, int* TW) {
  int best = 0;
  *TR = *TW = 1;
  for (int tr = 1; tr <= Ho; ++tr)
    for (int tw = 1; tw <= Wo; ++tw) {
      const int ec = (tw - 1) * stride + 3;
      const int em = ((tr - 1) * stride + 3) * (ec + (ec & 1));
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

template <int CB, int S>
static void expand_dw_launch_cb(const ExpandDwArgs& a, int ds, hipStream_t st) {
  const dim3 grid((unsigned)a.blocks);
  switch (ds) {
    case 1: launch(expand_dw_kernel<CB, 1, S>, grid, dim3(256), 0, st, a); break;
    case 2: launch(expand_dw_kernel<CB, 2, S>, grid, dim3(256), 0, st, a); break;
    case 3: launch(expand_dw_kernel<CB, 3, S>, grid, dim3(256), 0, st, a); break;
    case 4: launch(expand_dw_kernel<CB, 4, S>, grid, dim3(256), 0, st, a); break;
    default: launch(expand_dw_kernel<CB, 5, S>, grid, dim3(256), 0, st, a); break;
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
  a.ECP = a.EC + (a.EC & 1);
  a.EM = a.ER * a.ECP;
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
  a.div_chunks = FastDiv::make(a.chunks);
  a.div_tw = FastDiv::make(a.tiles_w);
  a.div_th = FastDiv::make(a.tiles_h);
  a.div_ecp = FastDiv::make(a.ECP);
  a.div_twi = FastDiv::make(stride == 1 ? (a.TW + 1) / 2 : a.TW);
  const int ds = ceil_div(Cin, 32);
  if (cb == 64)
    stride == 1 ? expand_dw_launch_cb<64, 1>(a, ds, st) : expand_dw_launch_cb<64, 2>(a, ds, st);
  else
    stride == 1 ? expand_dw_launch_cb<48, 1>(a, ds, st) : expand_dw_launch_cb<48, 2>(a, ds, st);
  DS_HIP(hipGetLastError());
  return DSTACK_OK;
}

}  // namespace dstack

