// Direct convolution of a 3-channel (RGB) image: the stems of the CNNs of
// Sec. 3 (ResNet-50 7x7/2 -> 64, MobileNetV2 3x3/2 -> 32, the tiny CNN's
// 3x3/1 -> 16), fused with scale, shift and activation, on the matrix cores.
//
// The image is read as it is (no packing to 8 channels in HBM).  A block
// takes 256 consecutive output pixels of one image; the input rows they touch
// are copied to LDS once, each pixel widened to 4 channels (8 bytes, channel
// 3 zero).  The GEMM depth is (window position q, channel c) with c in 0..3,
// so one MFMA depth step of 32 covers 8 window positions and a lane's
// 8-value fragment is two whole pixels: two 8-byte LDS reads for the image
// operand, one 16-byte load of the [K][R][R][4] weights (channel 3 zero) for
// the weight operand.  The weight fragments stay in registers for the whole
// block; each wave runs 4 groups of 16 pixels through v_mfma_f32_16x16x32_bf16
// (rows = output channels, columns = pixels) and stores each lane's 4
// consecutive channels of one pixel as an 8-byte vector.
#include <algorithm>

#include "common.hpp"

namespace dstack {

constexpr int RGB_PIX = 256;  // output pixels per block

template <int R, int K>
__global__ __launch_bounds__(256) void conv_rgb_kernel(const uint16_t* __restrict__ x, int H, int W,
                                                       const bf16* __restrict__ w4, int stride, int pad,
                                                       const float* __restrict__ scale,
                                                       const float* __restrict__ shift, int act, bf16* __restrict__ y,
                                                       int Ho, int Wo, int tiles_per_img, int vec16, int patch_bytes) {
  constexpr int RR = R * R;
  constexpr int DC = (RR + 7) / 8;  // depth steps of 8 window positions
  constexpr int KB = K / 16;        // 16-channel MFMA row blocks
  constexpr int ROW = K * 2 + 16;   // staged output row (one pixel), padded against bank conflicts
  extern __shared__ __attribute__((aligned(16))) unsigned char smem[];
  __shared__ __attribute__((aligned(16))) float bnl[2 * K];  // scale, shift
  uint2* patch = reinterpret_cast<uint2*>(smem);                // [rows][W] pixels, 4 bf16 each
  uint2* wl = reinterpret_cast<uint2*>(smem + patch_bytes);     // [K][RR] weight pixels, 4 bf16 each
  unsigned char* ot = smem + patch_bytes;  // after the weights are in registers: the output tile

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n = blockIdx.x / tiles_per_img;
  const int p0 = (blockIdx.x - n * tiles_per_img) * RGB_PIX;
  const int npix = Ho * Wo;
  const int p_last = min(p0 + RGB_PIX, npix) - 1;
  // input rows [lo, hi] of image n feed this block's outputs
  const int lo = max(0, (p0 / Wo) * stride - pad);
  const int hi = min(H - 1, (p_last / Wo) * stride - pad + R - 1);
  const long base = ((long)n * H + lo) * W * 3;  // first element
  const int cpx = (hi - lo + 1) * W;             // pixels in the patch

  // Stage the weights (K * RR 8-byte groups), the BN vectors and the patch
  // (widened to 4 channels) in LDS.  Every global load of a round is issued
  // before its LDS stores, so a block waits for one memory round trip (two
  // patch passes per round) rather than one per loop iteration.
  constexpr int WPT = (K * RR + 255) / 256;  // weight groups per thread
  {
    const uint2* wsrc = reinterpret_cast<const uint2*>(w4);
    uint2 wv[WPT];
#pragma unroll
    for (int i = 0; i < WPT; ++i) {
      const int idx = tid + i * 256;
      wv[i] = idx < K * RR ? wsrc[idx] : uint2{0u, 0u};
    }
    const float bv = tid < 2 * K ? (tid < K ? scale[tid] : shift[tid - K]) : 0.0f;
    if (vec16) {  // W % 8 == 0, 16-byte aligned image: 8 pixels = 3 16-byte loads -> 4 16-byte LDS writes
      const uint4* src = reinterpret_cast<const uint4*>(x + base);
      uint4* dst = reinterpret_cast<uint4*>(smem);
      const int n8 = cpx / 8;
      for (int g0 = tid; g0 < n8; g0 += 2 * 256) {
        uint4 v[2][3];
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int g8 = min(g0 + u * 256, n8 - 1);
#pragma unroll
          for (int e = 0; e < 3; ++e) v[u][e] = src[3 * g8 + e];
        }
        if (g0 == tid) {  // first pass: the weights and BN go to LDS while the patch loads are in flight
#pragma unroll
          for (int i = 0; i < WPT; ++i)
            if (tid + i * 256 < K * RR) wl[tid + i * 256] = wv[i];
          if (tid < 2 * K) bnl[tid] = bv;
        }
#pragma unroll
        for (int u = 0; u < 2; ++u) {
          const int g8 = g0 + u * 256;
          if (g8 >= n8) break;
          const uint32_t d[12] = {v[u][0].x, v[u][0].y, v[u][0].z, v[u][0].w, v[u][1].x, v[u][1].y,
                                  v[u][1].z, v[u][1].w, v[u][2].x, v[u][2].y, v[u][2].z, v[u][2].w};
          uint32_t w[16];  // pixel j -> (c0 | c1 << 16, c2)
#pragma unroll
          for (int j = 0; j < 8; ++j) {
            const int e = 3 * j;  // first element of pixel j; dword e / 2
            if ((j & 1) == 0) {
              w[2 * j] = d[e / 2];
              w[2 * j + 1] = d[e / 2 + 1] & 0xffffu;
            } else {
              w[2 * j] = (d[e / 2] >> 16) | (d[e / 2 + 1] << 16);
              w[2 * j + 1] = d[e / 2 + 1] >> 16;
            }
          }
#pragma unroll
          for (int q = 0; q < 4; ++q) dst[4 * g8 + q] = uint4{w[4 * q], w[4 * q + 1], w[4 * q + 2], w[4 * q + 3]};
        }
      }
      if (tid >= n8) {  // no patch pass ran on this thread
#pragma unroll
        for (int i = 0; i < WPT; ++i)
          if (tid + i * 256 < K * RR) wl[tid + i * 256] = wv[i];
        if (tid < 2 * K) bnl[tid] = bv;
      }
    } else {
      for (int i0 = tid; i0 < cpx; i0 += 256 * 4) {
        uint32_t c0[4], c1[4], c2[4];
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int i = min(i0 + u * 256, cpx - 1);
          c0[u] = x[base + 3L * i];
          c1[u] = x[base + 3L * i + 1];
          c2[u] = x[base + 3L * i + 2];
        }
#pragma unroll
        for (int u = 0; u < 4; ++u)
          if (i0 + u * 256 < cpx) patch[i0 + u * 256] = uint2{c0[u] | (c1[u] << 16), c2[u]};
      }
#pragma unroll
      for (int i = 0; i < WPT; ++i)
        if (tid + i * 256 < K * RR) wl[tid + i * 256] = wv[i];
      if (tid < 2 * K) bnl[tid] = bv;
    }
  }
  __syncthreads();

  // weight fragments: row k = kb*16 + lane%16, window positions q0, q0+1
  const int quad = lane >> 4;
  bf16x8 a[KB][DC];
#pragma unroll
  for (int kb = 0; kb < KB; ++kb)
#pragma unroll
    for (int dc = 0; dc < DC; ++dc) {
      const int q0 = dc * 8 + quad * 2;
      const int k = kb * 16 + (lane & 15);
      const uint2 v0 = q0 < RR ? wl[k * RR + q0] : uint2{0u, 0u};
      const uint2 v1 = q0 + 1 < RR ? wl[k * RR + q0 + 1] : uint2{0u, 0u};
      a[kb][dc] = __builtin_bit_cast(bf16x8, uint4{v0.x, v0.y, v1.x, v1.y});
    }
  __syncthreads();  // the weight area becomes the output tile [256 pixels][K] (rows padded to ROW bytes)

  const float lo_clamp = act == ACT_NONE ? -INFINITY : 0.0f, hi_clamp = act == ACT_RELU6 ? 6.0f : INFINITY;
  // patch offset (r * W + s) of this lane's window positions q = dc*8 +
  // quad*2 + h, and whether q is a real position (the depth tail is zero)
  int qoff[DC][2];
  unsigned qreal = 0;
#pragma unroll
  for (int dc = 0; dc < DC; ++dc)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int q = dc * 8 + quad * 2 + h;
      const int r = q / R, s = q - (q / R) * R;
      qoff[dc][h] = q < RR ? r * W + s : 0;
      if (q < RR) qreal |= 1u << (dc * 2 + h);
    }
#pragma unroll 1
  for (int g = 0; g < 4; ++g) {
    const int p = p0 + wave * 64 + g * 16 + (lane & 15);
    const int pc = min(p, p_last);
    const int ho = pc / Wo, wo = pc - (pc / Wo) * Wo;
    const int hr0 = ho * stride - pad, ws0 = wo * stride - pad;
    bf16x8 b[DC];
    // windows wholly inside the image (wave-uniform test): no per-position checks
    const bool inner = hr0 >= 0 && hr0 + R <= H && ws0 >= 0 && ws0 + R <= W;
    if (__ballot(inner) == ~0ull) {
      const uint2* pp = patch + (hr0 - lo) * W + ws0;
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) {
        uint2 v[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          v[h] = pp[qoff[dc][h]];
          if (dc * 8 + 8 > RR && !((qreal >> (dc * 2 + h)) & 1u)) v[h] = uint2{0u, 0u};
        }
        b[dc] = __builtin_bit_cast(bf16x8, uint4{v[0].x, v[0].y, v[1].x, v[1].y});
      }
    } else {
#pragma unroll
      for (int dc = 0; dc < DC; ++dc) {
        uint2 v[2];
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int q = dc * 8 + quad * 2 + h;
          const int r = q / R, s = q - (q / R) * R;
          const int hr = hr0 + r, ws = ws0 + s;
          const bool ok = q < RR && (unsigned)hr < (unsigned)H && (unsigned)ws < (unsigned)W;
          v[h] = ok ? patch[(hr - lo) * W + ws] : uint2{0u, 0u};
        }
        b[dc] = __builtin_bit_cast(bf16x8, uint4{v[0].x, v[0].y, v[1].x, v[1].y});
      }
    }
    // depth outer, channel blocks inner: KB independent accumulation chains in flight
    f32x4 accs[KB];
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) accs[kb] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int dc = 0; dc < DC; ++dc)
#pragma unroll
      for (int kb = 0; kb < KB; ++kb) accs[kb] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[kb][dc], b[dc], accs[kb], 0, 0, 0);
#pragma unroll
    for (int kb = 0; kb < KB; ++kb) {
      const f32x4 acc = accs[kb];
      const f32x4 sc = *reinterpret_cast<const f32x4*>(bnl + kb * 16 + 4 * quad);
      const f32x4 sh = *reinterpret_cast<const f32x4*>(bnl + K + kb * 16 + 4 * quad);
      bf16x4 o;  // this lane's channels kb*16 + 4*quad.. of its pixel
#pragma unroll
      for (int i = 0; i < 4; ++i) o[i] = (bf16)__builtin_amdgcn_fmed3f(acc[i] * sc[i] + sh[i], lo_clamp, hi_clamp);
      *reinterpret_cast<bf16x4*>(ot + (wave * 64 + g * 16 + (lane & 15)) * ROW + (kb * 16 + 4 * quad) * 2) = o;
    }
  }
  // the block's pixels are one contiguous run of the output: 16-byte vectors
  __syncthreads();
  constexpr int CPP = K / 8;  // 16-byte chunks per pixel
  const int chunks = (p_last - p0 + 1) * CPP;
  uint4* out = reinterpret_cast<uint4*>(y + ((long)n * npix + p0) * K);
  for (int c = tid; c < chunks; c += 256) {
    const int px = c / CPP, off = c - px * CPP;
    out[c] = *reinterpret_cast<const uint4*>(ot + px * ROW + off * 16);
  }
}

template <int R, int K>
static dstack_status rgb_launch(const bf16* x, int N, int H, int W, const bf16* w4, int stride, int pad,
                                const float* scale, const float* shift, int act, bf16* y, int Ho, int Wo,
                                hipStream_t st) {
  // rows a tile of 256 output pixels can span, and the input rows they need;
  // after the patch: the weights, then (in the same bytes) the output tile
  const int out_rows = (RGB_PIX + Wo - 2) / Wo + 1;
  const long patch = ((long)((out_rows - 1) * stride + R) * W * 8 + 15) / 16 * 16;
  const long lds = patch + std::max((long)K * R * R * 8, (long)RGB_PIX * (K * 2 + 16));
  DS_CHECK(lds <= 64 * 1024, DSTACK_E_UNSUPPORTED, "conv2d_rgb: image rows too wide for the LDS tile");
  DS_CHECK(((uintptr_t)w4 & 7) == 0 && ((uintptr_t)y & 15) == 0 && ((uintptr_t)scale & 15) == 0 &&
               ((uintptr_t)shift & 15) == 0,
           DSTACK_E_INVALID, "conv2d_rgb: w4 must be 8-byte aligned; y, scale and shift 16-byte aligned");
  const int tiles = (Ho * Wo + RGB_PIX - 1) / RGB_PIX;
  launch(conv_rgb_kernel<R, K>, dim3((unsigned)(N * tiles)), dim3(256), (size_t)lds, st,
                     reinterpret_cast<const uint16_t*>(x), H, W, w4, stride, pad, scale, shift, act, y, Ho, Wo, tiles,
                     (W % 8 == 0 && ((uintptr_t)x & 15) == 0) ? 1 : 0, (int)patch);
  return DSTACK_OK;
}

dstack_status launch_conv2d_rgb(const bf16* x, int N, int H, int W, const bf16* w4, int K, int R, int stride, int pad,
                                const float* scale, const float* shift, int act, bf16* y, hipStream_t st) {
  DS_CHECK(N > 0 && H > 0 && W > 0 && stride > 0 && pad >= 0 && pad < R, DSTACK_E_INVALID, "conv2d_rgb: bad shape");
  DS_CHECK(scale && shift, DSTACK_E_INVALID, "conv2d_rgb: scale and shift are required");
  const bool ok = (R == 3 && (K == 16 || K == 32 || K == 64)) || (R == 7 && K == 64);
  DS_CHECK(ok, DSTACK_E_UNSUPPORTED, "conv2d_rgb: supported (R, K): (3, 16), (3, 32), (3, 64), (7, 64)");
  const int Ho = out_dim(H, R, stride, pad), Wo = out_dim(W, R, stride, pad);
  DS_CHECK(Ho > 0 && Wo > 0, DSTACK_E_INVALID, "conv2d_rgb: empty output");
  DS_CHECK((long)N * H * W * 3 < (1L << 31) && (long)N * Ho * Wo * K < (1L << 31), DSTACK_E_UNSUPPORTED,
           "conv2d_rgb: tensor too large");
  dstack_status s;
  if (R == 7)
    s = rgb_launch<7, 64>(x, N, H, W, w4, stride, pad, scale, shift, act, y, Ho, Wo, st);
  else if (K == 16)
    s = rgb_launch<3, 16>(x, N, H, W, w4, stride, pad, scale, shift, act, y, Ho, Wo, st);
  else if (K == 32)
    s = rgb_launch<3, 32>(x, N, H, W, w4, stride, pad, scale, shift, act, y, Ho, Wo, st);
  else
    s = rgb_launch<3, 64>(x, N, H, W, w4, stride, pad, scale, shift, act, y, Ho, Wo, st);
  if (s != DSTACK_OK) return s;
  DS_HIP(hipGetLastError());
  return DSTACK_OK;
}

}  // namespace dstack
