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
// needs C % 8 == 0 (3-channel stems run in the direct RGB kernel instead).
//
// Data movement.  Each depth tile (BK = 64) of both operands is copied from
// global memory straight into LDS with buffer_load_dwordx4 ... lds: a wave's
// load moves 64 lanes x 16 bytes into one contiguous 1 KB LDS block (8 tile
// rows of 128 bytes).  An out-of-range buffer offset deposits zeros, which
// implements the convolution's zero padding, the pixel tail and the depth
// tail without branches on the data path.  A ring of STAGES such tiles keeps
// STAGES-1 tiles in flight while the matrix cores work on the current one;
// the wait is a vmcnt count (loads retire in order) followed by one barrier.
// Rows are stored unpadded with their eight 16-byte chunks XOR-swizzled by
// (row/2) % 8, so the 16 rows an MFMA fragment read touches fall on 16
// distinct 4-bank groups.
//
// Compute.  256 threads = 4 waves in a WN x WM grid over the (BN x BM) tile;
// each wave issues v_mfma_f32_16x16x32_bf16 on its (BN/WN x BM/WM) sub-tile.
// Operand layouts (checked on the device): lane l holds A[l%16][8*(l/16)..+8)
// and B[8*(l/16)..+8)[l%16]; the result holds C[4*(l/16)+i][l%16], i = 0..3,
// so each lane ends with 4 consecutive output channels of one pixel and the
// epilogue (scale, shift, residual, activation) is one 8-byte store.
//
// Split-K: with gridDim.z = splits > 1 each z-slice accumulates a range of
// depth tiles and writes raw fp32 partial sums to a workspace; the last block
// of each tile to finish (a per-tile arrival counter) sums the slices and
// applies the epilogue, so no second kernel is launched.
#include <hip/hip_ext.h>

#include <mutex>
#include <type_traits>

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
  unsigned* counters;  // split-K: per-tile arrival counters (zero between launches)
  int N, H, W, C, K, R, S, stride, pad, Ho, Wo;
  int M, Kg;
  int act;
  int kt_per_split;
  int tiles_n;         // output-channel tiles (fastest-varying in the tile order)
  int tiles;           // tiles per split slice
  int n_cu;            // CUs of the launch's partition (host-side planning only)
  FastDiv div_wo, div_ho, div_c, div_s, div_tn;
};

constexpr int BK = 64;          // depth per LDS stage (bf16 elements)
constexpr int ROW_BYTES = 128;  // one tile row = BK bf16
constexpr unsigned OOB = 0x80000000u;  // buffer offset past any tensor (< 2 GB): loads zeros
constexpr int CPOL_SC1 = 16;           // buffer cache-policy bit: device scope (past the per-XCD L2)

// Addressing of the activation operand: 1x1 stride 1 (the pixel row is the
// input row), 1x1 strided, C % 64 == 0 (a depth tile lies in one (r, s)), or
// the general per-chunk (r, s, c) decomposition.
enum ConvMode { MODE_1X1 = 0, MODE_TILED = 1, MODE_GENERIC = 2, MODE_1X1S1 = 3 };

__device__ __forceinline__ void store_out4(void* y, bool f32, long idx, const float v[4]) {
  if (f32) {
    f32x4 o = {v[0], v[1], v[2], v[3]};
    *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(y) + idx) = o;
  } else {
    bf16x4 o = {(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3]};
    *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(y) + idx) = o;
  }
}

// vmcnt wait with an immediate count (gfx9 encoding: vmcnt[3:0] | vmcnt[5:4] << 14,
// expcnt and lgkmcnt left at "no wait").
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

typedef __attribute__((__vector_size__(4 * sizeof(int)))) int i32x4;

// Raw buffer descriptor: base, no stride, num_records = byte size (offsets at
// or past it read as zero), gfx9 data-format word.
__device__ __forceinline__ i32x4 make_rsrc(const void* base, unsigned bytes) {
  const unsigned long long p = (unsigned long long)base;
  i32x4 r;
  r[0] = (int)(unsigned)(p & 0xffffffffu);
  r[1] = (int)(unsigned)((p >> 32) & 0xffffu);
  r[2] = (int)bytes;
  r[3] = 0x00020000;
  return r;
}

// 32-bit LDS byte address of a pointer into a __shared__ array.
__device__ __forceinline__ unsigned lds_address(const void* p) {
  return (unsigned)(unsigned long long)(const __attribute__((address_space(3))) void*)p;
}

// NL wave-loads of 16 bytes per lane: load j moves buffer offsets off[j]
// into LDS at lds_base + 1024 * j + 16 * lane.  Issued as inline asm so that
// the compiler does not treat every later LDS read as dependent on it (it
// would wait for all loads in flight); the kernel's own vmcnt waits order
// these loads against the LDS reads.  M0 (the LDS destination) is saved once,
// stepped by 1 KB between loads (one wait state after each write), restored.
template <int NL>
__device__ __forceinline__ void load_group(i32x4 rsrc, const unsigned (&off)[NL], unsigned lds_base);

template <>
__device__ __forceinline__ void load_group<1>(i32x4 rsrc, const unsigned (&off)[1], unsigned lds_base) {
  unsigned saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %2, %3, 0 offen lds\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds_base), "v"(off[0]), "s"(rsrc)
      : "memory");
}

template <>
__device__ __forceinline__ void load_group<2>(i32x4 rsrc, const unsigned (&off)[2], unsigned lds_base) {
  unsigned saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %2, %4, 0 offen lds\n\t"
      "s_add_u32 m0, m0, 0x400\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %3, %4, 0 offen lds\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds_base), "v"(off[0]), "v"(off[1]), "s"(rsrc)
      : "memory", "scc");
}

template <>
__device__ __forceinline__ void load_group<4>(i32x4 rsrc, const unsigned (&off)[4], unsigned lds_base) {
  unsigned saved;
  asm volatile(
      "s_mov_b32 %0, m0\n\t"
      "s_mov_b32 m0, %1\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %2, %6, 0 offen lds\n\t"
      "s_add_u32 m0, m0, 0x400\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %3, %6, 0 offen lds\n\t"
      "s_add_u32 m0, m0, 0x400\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %4, %6, 0 offen lds\n\t"
      "s_add_u32 m0, m0, 0x400\n\t"
      "s_nop 0\n\t"
      "buffer_load_dwordx4 %5, %6, 0 offen lds\n\t"
      "s_mov_b32 m0, %0"
      : "=&s"(saved)
      : "s"(lds_base), "v"(off[0]), "v"(off[1]), "v"(off[2]), "v"(off[3]), "s"(rsrc)
      : "memory", "scc");
}

template <int BN, int BM, int WN, int WM, int STAGES, int MODE, bool OUT_F32, bool SPLIT>
__global__ __launch_bounds__(256) void conv_igemm_kernel(ConvArgs a) {
  constexpr int ROWS = BN + BM;
  constexpr int STAGE_BYTES = ROWS * ROW_BYTES;
  constexpr int LPW = ROWS / 32;        // wave-loads (8 rows each) per wave per stage
  constexpr int TN = BN / WN / 16;      // MFMA tiles per wave along channels
  constexpr int TM = BM / WM / 16;      // ... along pixels
  static_assert(BN % 32 == 0 && BM % 32 == 0 && WN * WM == 4 && TN >= 1 && TM >= 1, "tile shape");
  static_assert(STAGES >= 2 && STAGES <= 4, "2..4 stages");

  __shared__ __attribute__((aligned(1024))) unsigned char lds[STAGES * STAGE_BYTES];

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wn = wave % WN, wm = wave / WN;
  // XCD-aware tile order: consecutive workgroups go round-robin to the 8 XCDs,
  // so XCD x is given the contiguous tile range [x*q + min(x, r), ...) of the
  // (pixel tile, channel tile) order with channel tiles fastest; the blocks
  // that share an activation tile then share that XCD's L2.
  int tile;
  {
    const int L = blockIdx.x;
    const int q = a.tiles >> 3, r = a.tiles & 7;
    const int x = L & 7, i = L >> 3;
    tile = x * q + min(x, r) + i;
  }
  const int tm_idx = a.div_tn.div(tile);
  const int n0 = (tile - tm_idx * a.tiles_n) * BN;
  const int m0 = tm_idx * BM;

  const i32x4 wrs = make_rsrc(a.w, (unsigned)((long)a.K * a.Kg * 2));
  const i32x4 xrs = make_rsrc(a.x, (unsigned)((long)a.N * a.H * a.W * a.C * 2));
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);  // wave-uniform copy: scalar branches
  const unsigned lds0 = __builtin_amdgcn_readfirstlane(lds_address(lds));

  // ---- per-lane addressing ----
  // Every wave moves WPW 8-row groups of weight rows and APW 8-row groups of
  // pixel rows per stage; lane l moves 16-byte chunk (l % 8) of row l / 8 of
  // each group, stored at its swizzled position.
  constexpr int WPW = BN / 32, APW = BM / 32;
  const int rin = lane >> 3;
  unsigned woff[WPW];  // byte offset of the lane's chunk at depth 0; OOB past K (stays >= 2^31 after adding depth)
#pragma unroll
  for (int j = 0; j < WPW; ++j) {
    const int r = 8 * (wave * WPW + j) + rin;
    const int c = (lane & 7) ^ ((r >> 1) & 7);
    const int n = n0 + r;
    woff[j] = n < a.K ? (unsigned)(((long)n * a.Kg + c * 8) * 2) : OOB;
  }
  // pixel rows: 1x1 modes keep the chunk's byte offset at depth 0 (OOB past
  // M); TILED keeps the byte offset of the chunk at (r, s) = (0, 0) relative
  // to the (possibly padded-out) top-left input pixel, plus a bit mask of the
  // (r, s) window positions that fall inside the image; GENERIC keeps the
  // image's first pixel and the top-left coordinate.
  int aoff[APW];
  unsigned vmask[APW];
  int hi0[APW], wi0[APW], chunk[APW];
#pragma unroll
  for (int j = 0; j < APW; ++j) {
    const int rl = 8 * (wave * APW + j) + rin;
    const int r = BN + rl;
    const int c = (lane & 7) ^ ((r >> 1) & 7);
    chunk[j] = c;
    const int m = m0 + rl;
    aoff[j] = (int)OOB;
    vmask[j] = 0;
    hi0[j] = 0;
    wi0[j] = 0;
    if (m < a.M) {
      const int t = a.div_wo.div(m);
      const int wo = m - t * a.Wo;
      const int nn = a.div_ho.div(t);
      const int ho = t - nn * a.Ho;
      if (MODE == MODE_1X1S1) {  // the output pixel is the input pixel
        aoff[j] = (int)(((long)m * a.C + c * 8) * 2);
      } else if (MODE == MODE_1X1) {
        aoff[j] = (int)(((((long)nn * a.H + ho * a.stride) * a.W + wo * a.stride) * a.C + c * 8) * 2);
      } else {
        const int h0 = ho * a.stride - a.pad, w0 = wo * a.stride - a.pad;
        if (MODE == MODE_TILED) {
          aoff[j] = ((((nn * a.H + h0) * a.W + w0) * a.C) + c * 8) * 2;
          // window rows [rlo, rhi) and columns [slo, shi) fall inside the image
          const int rlo = max(0, -h0), rhi = min(a.R, a.H - h0);
          const int slo = max(0, -w0), shi = min(a.S, a.W - w0);
          const unsigned cols = shi > slo ? (unsigned)((1ull << shi) - (1ull << slo)) : 0u;  // S <= 32
          for (int rr = 0; rr < a.R; ++rr)
            if (rr >= rlo && rr < rhi) vmask[j] |= cols << (rr * a.S);
        } else {
          aoff[j] = nn * a.H * a.W;  // image's first pixel
          vmask[j] = 1;
          hi0[j] = h0;
          wi0[j] = w0;
        }
      }
    }
  }

  const int nkt_total = (a.Kg + BK - 1) / BK;
  int kt0 = 0, kt1 = nkt_total;
  if (SPLIT) {
    kt0 = blockIdx.z * a.kt_per_split;
    kt1 = min(nkt_total, kt0 + a.kt_per_split);
  }
  const bool kfull = (a.Kg % BK) == 0;  // no depth tail

  // issue the direct-to-LDS loads of depth tile kt into stage `st`.  Weight
  // chunks past the depth Kg read the next row (finite values) or zeros; the
  // pixel chunks there are forced to zero, so they add nothing.
  auto issue = [&](int kt, int st) {
    const int k0 = kt * BK;
    const unsigned sb = lds0 + st * STAGE_BYTES;
    unsigned wv[WPW];
#pragma unroll
    for (int j = 0; j < WPW; ++j) wv[j] = woff[j] + (unsigned)(k0 * 2);
    load_group<WPW>(wrs, wv, sb + wave_u * WPW * 1024);
    unsigned av[APW];
    if (MODE == MODE_1X1 || MODE == MODE_1X1S1) {
#pragma unroll
      for (int j = 0; j < APW; ++j) {
        const bool kin = kfull || k0 + chunk[j] * 8 < a.Kg;
        av[j] = kin ? (unsigned)aoff[j] + (unsigned)(k0 * 2) : OOB;
      }
    } else if (MODE == MODE_TILED) {  // C % 64 == 0: the whole tile is inside one (r, s)
      const int rs = a.div_c.div(k0);
      const int tc = k0 - rs * a.C;
      const int tr = a.div_s.div(rs);
      const int ts = rs - tr * a.S;
      const int delta = ((tr * a.W + ts) * a.C + tc) * 2;  // wave-uniform
#pragma unroll
      for (int j = 0; j < APW; ++j) av[j] = ((vmask[j] >> rs) & 1) ? (unsigned)(aoff[j] + delta) : OOB;
    } else {
#pragma unroll
      for (int j = 0; j < APW; ++j) {
        const int k = k0 + chunk[j] * 8;
        const int rs = a.div_c.div(k);
        const int c = k - rs * a.C;
        const int r = a.div_s.div(rs);
        const int s = rs - r * a.S;
        const int hi = hi0[j] + r, wi = wi0[j] + s;
        const bool ok = vmask[j] && k < a.Kg && (unsigned)hi < (unsigned)a.H && (unsigned)wi < (unsigned)a.W;
        av[j] = ok ? (unsigned)(((aoff[j] + hi * a.W + wi) * a.C + c) * 2) : OOB;
      }
    }
    load_group<APW>(xrs, av, sb + (BN / 8 + wave_u * APW) * 1024);
  };

  f32x4 acc[TN][TM];
#pragma unroll
  for (int i = 0; i < TN; ++i)
#pragma unroll
    for (int j = 0; j < TM; ++j) acc[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};

  // fragment read addresses (bytes within a stage) for logical chunk `c` of row `r`
  auto frag = [&](const unsigned char* sb, int r, int c) -> bf16x8 {
    return *reinterpret_cast<const bf16x8*>(sb + r * ROW_BYTES + ((c ^ ((r >> 1) & 7)) << 4));
  };
  const int arow = wn * (BN / WN) + (lane & 15);
  const int brow = BN + wm * (BM / WM) + (lane & 15);
  const int cq = lane >> 4;

  // Epilogue mapping: thread -> fixed 4-channel group (256 is a multiple of
  // the groups per row) and ROWS_PT pixel rows RSTEP apart.  Its per-channel
  // scale and shift are fetched now and its residual rows right after the
  // last depth tile's loads, so that neither round trip follows the loop.
  constexpr int G = BN / 4;
  constexpr int RSTEP = 256 / G;
  constexpr int ROWS_PT = BM / RSTEP;
  static_assert(256 % G == 0 && BM % RSTEP == 0, "epilogue thread mapping");
  static_assert(2 * LPW + ROWS_PT < 64, "vmcnt range");
  const int cl = (tid % G) * 4;
  const int ch0 = n0 + cl;
  const int pl0 = tid / G;
  const int chc = min(ch0, a.K - 4);  // in-range channel for the prefetches (K % 4 == 0)
  f32x4 sc = f32x4{1.f, 1.f, 1.f, 1.f}, sh = f32x4{0.f, 0.f, 0.f, 0.f};
  if (!SPLIT || a.counters) {
    if (a.scale) sc = *reinterpret_cast<const f32x4*>(a.scale + chc);
    if (a.shift) sh = *reinterpret_cast<const f32x4*>(a.shift + chc);
  }
  // residual rows: exactly ROWS_PT buffer loads per lane (rows past M read
  // row M-1 and are not stored), so the stage waits can count them
  const bool has_res = !SPLIT && a.res != nullptr;
  bf16x4 rv[ROWS_PT];
  auto load_res = [&]() __attribute__((always_inline)) {
    const __amdgpu_buffer_rsrc_t rr =
        __builtin_amdgcn_make_buffer_rsrc((void*)a.res, (short)0, (int)(unsigned)((long)a.M * a.K * 2), 0x00020000);
#pragma unroll
    for (int k = 0; k < ROWS_PT; ++k) {
      const int px = min(m0 + pl0 + k * RSTEP, a.M - 1);
      const auto v = __builtin_amdgcn_raw_buffer_load_b64(rr, (int)(((unsigned)px * (unsigned)a.K + (unsigned)chc) * 2u), 0, 0);
      rv[k] = __builtin_bit_cast(bf16x4, v);
    }
  };
#pragma unroll
  for (int k = 0; k < ROWS_PT; ++k) rv[k] = bf16x4{};

  // prologue: STAGES-1 tiles in flight
#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s)
    if (kt0 + s < kt1) issue(kt0 + s, s);
  if (has_res && kt1 - kt0 <= STAGES - 1) load_res();

  for (int kt = kt0; kt < kt1; ++kt) {
    const int st = (kt - kt0) % STAGES;
    // tiles issued after kt that may stay in flight
    // (the residual rows, once issued, are the youngest loads)
    const int after = min(STAGES - 2, kt1 - 1 - kt);
    if (has_res && kt1 - 1 - kt <= STAGES - 2) {
      if (after >= 2)
        wait_vmcnt<2 * LPW + ROWS_PT>();
      else if (after == 1)
        wait_vmcnt<LPW + ROWS_PT>();
      else
        wait_vmcnt<ROWS_PT>();
    } else {
      if (after >= 2)
        wait_vmcnt<2 * LPW>();
      else if (after == 1)
        wait_vmcnt<LPW>();
      else
        wait_vmcnt<0>();
    }
    __syncthreads();  // every wave's part of tile kt is in LDS; every wave is done with tile kt-1
    if (kt + STAGES - 1 < kt1) {
      issue(kt + STAGES - 1, (kt - kt0 + STAGES - 1) % STAGES);
      if (has_res && kt + STAGES - 1 == kt1 - 1) load_res();
    }
    const unsigned char* sb = lds + st * STAGE_BYTES;
#pragma unroll
    for (int ks = 0; ks < BK / 8; ks += 4) {
      bf16x8 af[TN], bfr[TM];
#pragma unroll
      for (int i = 0; i < TN; ++i) af[i] = frag(sb, arow + i * 16, ks + cq);
#pragma unroll
      for (int j = 0; j < TM; ++j) bfr[j] = frag(sb, brow + j * 16, ks + cq);
#pragma unroll
      for (int i = 0; i < TN; ++i)
#pragma unroll
        for (int j = 0; j < TM; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
    }
  }

  // Epilogue through LDS: each lane holds channels ch..ch+3 of one pixel per
  // MFMA tile, i.e. 8-byte pieces of 16 different pixel rows.  The fp32 tile
  // is first written to LDS as [pixel][channel] (unpadded rows of BN floats,
  // 16-byte units XOR-swizzled by pixel % 8), then consecutive threads take
  // consecutive 4-channel groups of a pixel row, so residual reads and output
  // writes cover whole row segments.
  static_assert(BM * BN * 4 <= STAGES * STAGE_BYTES, "epilogue tile must fit in the stage ring");
  static_assert(BN / 4 >= 8, "swizzle needs 8 units per row");
  wait_vmcnt<0>();  // scale, shift and residual rows are in registers: no waits between the row stores
  __syncthreads();  // all waves are done reading the last stage
  float* ct = reinterpret_cast<float*>(lds);
  auto cidx = [](int pl, int cl) { return pl * BN + ((((cl >> 2) ^ (pl & 7))) << 2); };
#pragma unroll
  for (int i = 0; i < TN; ++i) {
    const int cl = wn * (BN / WN) + i * 16 + (lane >> 4) * 4;
#pragma unroll
    for (int j = 0; j < TM; ++j) {
      const int pl = wm * (BM / WM) + j * 16 + (lane & 15);
      *reinterpret_cast<f32x4*>(ct + cidx(pl, cl)) = acc[i][j];
    }
  }
  __syncthreads();
  // all of the thread's rows are read from LDS before the first store
  f32x4 t[ROWS_PT];
#pragma unroll
  for (int k = 0; k < ROWS_PT; ++k) t[k] = *reinterpret_cast<const f32x4*>(ct + cidx(pl0 + k * RSTEP, cl));
  if (SPLIT) {
    // Fused reduction: every block writes its slice with device-scope stores
    // (they pass the per-XCD L2s) and bumps the tile's counter once they have
    // all completed; the block that brings it to gridDim.z reads the slices
    // back in slice order (the sum does not depend on which block is last),
    // runs the epilogue and puts the counter back to 0 for the next launch.
    const unsigned slice_bytes = (unsigned)a.M * (unsigned)a.K * 4u;  // split workspaces are < 4 GB
    const __amdgpu_buffer_rsrc_t pa =
        __builtin_amdgcn_make_buffer_rsrc(a.partial, (short)0, (int)(slice_bytes * gridDim.z), 0x00020000);
    if (ch0 < a.K) {
#pragma unroll
      for (int k = 0; k < ROWS_PT; ++k) {
        const int px = m0 + pl0 + k * RSTEP;
        if (px < a.M)
          __builtin_amdgcn_raw_buffer_store_b128(
              t[k], pa, (int)(blockIdx.z * slice_bytes + ((unsigned)px * a.K + ch0) * 4u), 0, CPOL_SC1);
      }
    }
    wait_vmcnt<0>();
    __syncthreads();  // the whole slice is written; every thread is done reading the staged tile
    int* flag = reinterpret_cast<int*>(lds);
    if (tid == 0)
      *flag = (int)__hip_atomic_fetch_add(a.counters + tile, 1u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    __syncthreads();
    if (*flag != (int)gridDim.z - 1) return;
    if (tid == 0) __hip_atomic_store(a.counters + tile, 0u, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT);
    if (ch0 >= a.K) return;
    if (a.res && ROWS_PT < 16) load_res();  // in flight with the slices (128-pixel tiles: after them)
    const int S = gridDim.z;
    // ZC slices per round, all of their loads in flight together (64 VGPRs)
    constexpr int ZC = ROWS_PT >= 16 ? 1 : 16 / ROWS_PT;
    for (int z0 = 0; z0 < S; z0 += ZC) {
      f32x4 q[ZC][ROWS_PT];
#pragma unroll
      for (int c = 0; c < ZC; ++c) {
        const unsigned z = (unsigned)min(z0 + c, S - 1);
#pragma unroll
        for (int k = 0; k < ROWS_PT; ++k) {
          const int px = min(m0 + pl0 + k * RSTEP, a.M - 1);
          q[c][k] = __builtin_amdgcn_raw_buffer_load_b128(pa, (int)(z * slice_bytes + ((unsigned)px * a.K + ch0) * 4u),
                                                          0, CPOL_SC1);
        }
      }
#pragma unroll
      for (int c = 0; c < ZC; ++c)
        if (z0 + c < S)
#pragma unroll
          for (int k = 0; k < ROWS_PT; ++k) t[k] = z0 + c == 0 ? q[c][k] : t[k] + q[c][k];
    }
    if (a.res && ROWS_PT >= 16) load_res();
    wait_vmcnt<0>();  // residual rows
  }
  if (ch0 >= a.K) return;
  // element index of the thread's first row; rows step by RSTEP pixels
  // (M * K < 2^31 is checked at launch)
  const int idx0 = (m0 + pl0) * a.K + ch0;
  const int dstep = RSTEP * a.K;
  // the activation is chosen once: none, a clamp to [0, hi] (ReLU: hi =
  // inf), GELU or tanh
  const float hi = a.act == ACT_RELU6 ? 6.0f : INFINITY;
  auto rows = [&](auto act) {
#pragma unroll
    for (int k = 0; k < ROWS_PT; ++k) {
      if (m0 + pl0 + k * RSTEP >= a.M) continue;
      float v[4];
#pragma unroll
      for (int e = 0; e < 4; ++e) v[e] = act(t[k][e] * sc[e] + sh[e] + (float)rv[k][e]);
      store_out4(a.y, OUT_F32, idx0 + k * dstep, v);
    }
  };
  if (a.act == ACT_NONE)
    rows([](float v) { return v; });
  else if (a.act == ACT_GELU)
    rows([](float v) { return gelu_erf(v); });
  else if (a.act == ACT_TANH)
    rows([](float v) { return tanhf(v); });
  else
    rows([hi](float v) { return fminf(fmaxf(v, 0.0f), hi); });
}

// 256-thread launch; through hipExtLaunchKernelGGL when dispatch events are
// armed (and not while launch shapes are being recorded)
template <typename K, typename... Args>
static void launch_k(K kernel, dim3 grid, hipStream_t st, hipEvent_t e0, hipEvent_t e1, Args... args) {
  if ((e0 || e1) && !shape_recorder())
    hipExtLaunchKernelGGL(kernel, grid, dim3(256), 0, st, e0, e1, 0, args...);
  else
    launch(kernel, grid, dim3(256), 0, st, args...);
}

// 1x1, stride-1 convolution of small depth (C <= 32): a streaming GEMM that
// stages nothing of its inputs in LDS.  The output (M x K) is many times the
// input (M x C) and the weights (K x C) are tiny, so the layer is bound by
// writing its output.  Each wave keeps NB channel blocks (16 channels each)
// of weight fragments in registers (A operand; depth in KS steps of 32, zero
// past C) and walks pixel groups of 16: the group's B fragment is read
// straight from the input rows (lane l: pixel l % 16, depth 8 * (l / 16) ..
// + 8), and NB x KS MFMAs give each lane 4 consecutive channels of one pixel
// per block.  Scale and shift are applied there; with more than one block
// the fp32 tile then goes through the wave's own LDS region (rows padded by
// 16 bytes) so that each lane finishes 8 consecutive channels of one pixel:
// residual reads and output stores are 16-byte pieces of whole pixel rows.  The next group's
// fragment is loaded before the current one is multiplied.  Grid: x strides
// over pixel groups (4 waves per block), y over channel chunks of 16 * NB.
template <int NB, int KS, bool OUT_F32>
__global__ __launch_bounds__(256) void conv_igemm_1x1s_kernel(ConvArgs a, int groups) {
  constexpr int RS = 16 * NB + 4;  // staged row stride in floats
  __shared__ __attribute__((aligned(16))) float stage[4][16 * RS];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int row = lane & 15, kq = (lane >> 4) * 8;
  const int cb0 = blockIdx.y * NB;  // first 16-channel block of this chunk
  float* my = stage[wave];
  bf16x8 wa[NB][KS];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int ch = (cb0 + b) * 16 + row;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int k = s * 32 + kq;
      wa[b][s] = (ch < a.K && k < a.C) ? *reinterpret_cast<const bf16x8*>(a.w + (long)ch * a.C + k) : bf16x8{};
    }
  }
  // per-lane scale and shift of its 4 channels in every block, kept across groups
  f32x4 sc[NB], sh[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) {
    const int ch0 = (cb0 + b) * 16 + 4 * (lane >> 4);
    const bool in = ch0 < a.K;
    sc[b] = (in && a.scale) ? *reinterpret_cast<const f32x4*>(a.scale + ch0) : f32x4{1.f, 1.f, 1.f, 1.f};
    sh[b] = (in && a.shift) ? *reinterpret_cast<const f32x4*>(a.shift + ch0) : f32x4{0.f, 0.f, 0.f, 0.f};
  }
  const bool clamp = a.act != ACT_NONE;
  const float hi = a.act == ACT_RELU6 ? 6.0f : INFINITY;
  auto load_px = [&](int g, bf16x8 (&bx)[KS]) {
    const int px = g * 16 + row;
#pragma unroll
    for (int s = 0; s < KS; ++s) {
      const int k = s * 32 + kq;
      bx[s] = (g < groups && px < a.M && k < a.C) ? *reinterpret_cast<const bf16x8*>(a.x + (long)px * a.C + k)
                                                  : bf16x8{};
    }
  };
  const int stride = gridDim.x * 4;
  int g = blockIdx.x * 4 + wave;
  bf16x8 cur[KS], nxt[KS];
  load_px(g, cur);
  for (; g < groups; g += stride) {
    load_px(g + stride, nxt);
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < KS; ++s) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(wa[b][s], cur[s], acc, 0, 0, 0);
      // C layout: lane holds channels 4 * (lane / 16) + i of block b, pixel lane % 16
      f32x4 t;
#pragma unroll
      for (int i = 0; i < 4; ++i) t[i] = acc[i] * sc[b][i] + sh[b][i];
      if (NB == 1) {  // 16-channel rows: the 64 lanes' 8-byte pieces already tile whole rows
        const int px = g * 16 + row, ch0 = cb0 * 16 + 4 * (lane >> 4);
        if (px < a.M && ch0 < a.K) {
          const int idx = px * a.K + ch0;
          const bf16x4 r4 = a.res ? *reinterpret_cast<const bf16x4*>(a.res + idx) : bf16x4{};
          float v[4];
#pragma unroll
          for (int i = 0; i < 4; ++i) {
            const float u = t[i] + (float)r4[i];
            v[i] = clamp ? fminf(fmaxf(u, 0.0f), hi) : u;
          }
          store_out4(a.y, OUT_F32, idx, v);
        }
      } else {
        *reinterpret_cast<f32x4*>(my + row * RS + 16 * b + 4 * (lane >> 4)) = t;
      }
    }
    if (NB == 1) {
#pragma unroll
      for (int s = 0; s < KS; ++s) cur[s] = nxt[s];
      continue;
    }
    // the wave reads back what its own lanes wrote (LDS keeps a wave's order)
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    // 16 pixels x 2*NB pieces of 8 channels
#pragma unroll
    for (int p = 0; p < (32 * NB + 63) / 64; ++p) {
      const int e = p * 64 + lane;
      if (e >= 32 * NB) break;
      const int pl = e / (2 * NB), c8 = e - pl * (2 * NB);
      const int px = g * 16 + pl, ch = cb0 * 16 + 8 * c8;
      if (px >= a.M || ch >= a.K) continue;
      const f32x4 t0 = *reinterpret_cast<const f32x4*>(my + pl * RS + 8 * c8);
      const f32x4 t1 = *reinterpret_cast<const f32x4*>(my + pl * RS + 8 * c8 + 4);
      const int idx = px * a.K + ch;
      const bf16x8 r8 = a.res ? *reinterpret_cast<const bf16x8*>(a.res + idx) : bf16x8{};
      float v[8];
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        v[i] = t0[i] + (float)r8[i];
        v[i + 4] = t1[i] + (float)r8[i + 4];
      }
#pragma unroll
      for (int i = 0; i < 8; ++i) v[i] = clamp ? fminf(fmaxf(v[i], 0.0f), hi) : v[i];
      if (OUT_F32) {
        float* yo = reinterpret_cast<float*>(a.y) + idx;
        *reinterpret_cast<f32x4*>(yo) = f32x4{v[0], v[1], v[2], v[3]};
        *reinterpret_cast<f32x4*>(yo + 4) = f32x4{v[4], v[5], v[6], v[7]};
      } else {
        bf16x8 o;
#pragma unroll
        for (int i = 0; i < 8; ++i) o[i] = (bf16)v[i];
        *reinterpret_cast<bf16x8*>(reinterpret_cast<bf16*>(a.y) + idx) = o;
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
    for (int s = 0; s < KS; ++s) cur[s] = nxt[s];
  }
}

template <int NB, int KS>
static void launch_1x1s_nb(const ConvArgs& a, bool f32, int n_cu, hipStream_t st) {
  const int groups = ceil_div(a.M, 16);
  const int chunks = ceil_div(a.K, 16 * NB);
  // about 32 waves per CU over all chunks (their loads in flight hide the
  // latency of the next group); every wave walks >= 1 group
  const int bx = max(1, min(ceil_div(groups, 4), ceil_div(n_cu * 8, chunks)));
  const dim3 grid(bx, chunks);
  const DispatchEvents& de = dispatch_events();
  if (f32)
    launch_k(conv_igemm_1x1s_kernel<NB, KS, true>, grid, st, de.start, de.stop, a, groups);
  else
    launch_k(conv_igemm_1x1s_kernel<NB, KS, false>, grid, st, de.start, de.stop, a, groups);
}

// channel blocks per wave: the largest divisor of K / 16 that is at most 8
static void launch_1x1s(const ConvArgs& a, bool f32, int n_cu, hipStream_t st) {
  const int blocks = a.K / 16;
  int nb = 8;
  while (blocks % nb) --nb;
#define DS_NB_CASE(N)                   \
  case N:                               \
    launch_1x1s_nb<N, 1>(a, f32, n_cu, st); \
    break;
  switch (nb) {
    DS_NB_CASE(1)
    DS_NB_CASE(2)
    DS_NB_CASE(3)
    DS_NB_CASE(4)
    DS_NB_CASE(5)
    DS_NB_CASE(6)
    DS_NB_CASE(7)
    DS_NB_CASE(8)
  }
#undef DS_NB_CASE
}

struct ConvPlan {
  int bn, bm, splits;
};

// Tile and split choice from the GEMM shape and the CUs of the partition, by
// an estimate of the launch's duration.  Two blocks share a CU (the LDS ring
// is sized for it; more with the short ring), so a launch runs in
// ceil(blocks / (blocks per CU * CUs)) rounds and
// blocks of one round start and end together; a block costs a ramp until its
// first depth tile lands, a per-step time that depends on the tile shape, and
// an epilogue (plus, with a fused split-K, the wait for its slice to reach
// device scope and the last block's read-back of all slices).  The constants
// are per-block phase times measured on MI355X with two blocks per CU.  Split
// plans are considered only when the caller gives a workspace and counters.
struct TileCost {
  int bn, bm;
  double step_us;  // one 64-deep step
};
static constexpr TileCost kTiles[] = {
    {128, 128, 0.65}, {128, 64, 0.485}, {64, 128, 0.50}, {64, 64, 0.42}, {32, 128, 0.25}};
constexpr double kRampUs = 1.4;
constexpr double kSliceWriteUs = 2.6;   // device-scope slice stores until acknowledged
constexpr double kSliceReadUs = 0.75;   // per slice of 8192 fp32 values, the last block's read-back

// Launches whose blocks walk at most kShortTiles depth tiles (split-K
// slices: at most kShortSplitTiles) run with a two-tile ring, so that more
// blocks share a CU: as many as its 160 KB of LDS hold, at most as many as
// the registers allow (VGPR + AGPR per lane of the tile shapes).  Measured on
// MI355X (128 CUs): ResNet-50's 56x56 1x1 layers of depth 64 went from 19.3
// to 16.6 us and its 56x56 3x3 layers of 64 channels (9 depth tiles) from
// 17.8 to 15 us, MobileNetV2's 56x56 projections of depth 96 and 144 from
// 12.2 and 14.4 to 9.2 and 12.0 us; split plans of MobileNetV2's 7x7 layers
// were slower with the short ring beyond 3 tiles per slice.
constexpr int kShortTiles = 9;
constexpr int kShortSplitTiles = 3;
// (and only where the grid has more blocks than two per CU: a smaller grid
// gains nothing from the extra room and loses the deeper prefetch)
static bool short_ring(int per, int splits, long blocks, int n_cu) {
  return per <= (splits > 1 ? kShortSplitTiles : kShortTiles) && blocks > 2L * n_cu;
}
static int short_blocks_per_cu(int bn, int bm, bool split) {
  const int ring = 2 * (bn + bm) * ROW_BYTES;
  const int regs = bn * bm >= 16384 ? (split ? 240 : 200) : bn * bm >= 8192 ? (split ? 144 : 128) : (split ? 112 : 80);
  return max(1, min(160 * 1024 / ring, 512 / regs));
}

static double plan_cost(const TileCost& t, int M, int K, int nkt, int splits, int n_cu) {
  const int per = ceil_div(nkt, splits);
  const int s = ceil_div(nkt, per);
  const long blocks = (long)ceil_div(M, t.bm) * ceil_div(K, t.bn) * s;
  const long bpc = short_ring(per, s, blocks, n_cu) ? short_blocks_per_cu(t.bn, t.bm, s > 1) : 2;
  const long rounds = (blocks + bpc * n_cu - 1) / (bpc * n_cu);
  double blk = kRampUs + per * t.step_us + 0.6 + 1.5 * (t.bn * t.bm) / 16384.0;
  if (s > 1) blk += kSliceWriteUs + kSliceReadUs * s * (t.bn * t.bm) / 8192.0;
  return (double)rounds * blk;
}

static ConvPlan choose_plan(int M, int K, int Kg, int n_cu, bool can_split, size_t split_bytes) {
  // channel tiles: 32 for K <= 32, 64 for K <= 64, else 64 or 128
  const int bn_min = K <= 32 ? 32 : 64, bn_max = K <= 32 ? 32 : (K <= 64 ? 64 : 128);
  const int nkt = ceil_div(Kg, BK);
  ConvPlan best{bn_max, 128, 1};
  double best_t = 1e30;
  for (const TileCost& t : kTiles) {
    if (t.bn < bn_min || t.bn > bn_max) continue;
    for (int sp = 1; sp <= 16; sp *= 2) {
      if (sp > 1 && (!can_split || nkt / sp < 2 || (size_t)sp * M * K * sizeof(float) > split_bytes)) break;
      if (sp > 1 && (long)ceil_div(M, t.bm) * ceil_div(K, t.bn) > SPLITK_TILE_COUNTERS) break;
      const double c = plan_cost(t, M, K, nkt, sp, n_cu);
      if (c < best_t * 0.97) {  // a split or a smaller tile must win by more than 3%
        best_t = c;
        best = ConvPlan{t.bn, t.bm, sp};
      }
    }
  }
  return best;
}

size_t conv_splitk_workspace_bytes(int M, int K, int Kg, int n_cu) {
  ConvPlan p = choose_plan(M, K, Kg, n_cu, true, (size_t)1 << 40);
  return p.splits > 1 ? (size_t)p.splits * M * K * sizeof(float) : 0;
}

// Ring depth per tile shape: the deepest ring (at most 4) with which two
// blocks still share a CU's 160 KB of LDS, so that two blocks and STAGES-1
// tiles each keep loads in flight.
constexpr int conv_stages(int bn, int bm) {
  const int stage = (bn + bm) * ROW_BYTES;
  const int s = (80 * 1024) / stage;
  return s < 2 ? 2 : (s > 4 ? 4 : s);
}

template <int BN, int BM, int WN, int WM, int MODE>
static void launch_mode(ConvArgs a, bool f32, int splits, int stages, hipStream_t st) {
  constexpr int STAGES = conv_stages(BN, BM);
  a.tiles_n = ceil_div(a.K, BN);
  a.tiles = ceil_div(a.M, BM) * a.tiles_n;
  a.div_tn = FastDiv::make(a.tiles_n);
  dim3 grid(a.tiles, 1, splits);
  // with dispatch events armed: both on this kernel (the split-K reduction is in it)
  const DispatchEvents& de = dispatch_events();
  hipEvent_t e0 = de.start, e1 = de.stop;
  if (STAGES > 2 && stages == 2) {
    if (splits > 1)
      launch_k(conv_igemm_kernel<BN, BM, WN, WM, 2, MODE, false, true>, grid, st, e0, e1, a);
    else if (f32)
      launch_k(conv_igemm_kernel<BN, BM, WN, WM, 2, MODE, true, false>, grid, st, e0, e1, a);
    else
      launch_k(conv_igemm_kernel<BN, BM, WN, WM, 2, MODE, false, false>, grid, st, e0, e1, a);
  } else if (splits > 1)
    launch_k(conv_igemm_kernel<BN, BM, WN, WM, STAGES, MODE, false, true>, grid, st, e0, e1, a);
  else if (f32)
    launch_k(conv_igemm_kernel<BN, BM, WN, WM, STAGES, MODE, true, false>, grid, st, e0, e1, a);
  else
    launch_k(conv_igemm_kernel<BN, BM, WN, WM, STAGES, MODE, false, false>, grid, st, e0, e1, a);
}

template <int BN, int BM, int WN, int WM>
static void launch_cfg(const ConvArgs& a, int mode, bool f32, int splits, int stages, hipStream_t st) {
  if (mode == MODE_1X1S1)
    launch_mode<BN, BM, WN, WM, MODE_1X1S1>(a, f32, splits, stages, st);
  else if (mode == MODE_1X1)
    launch_mode<BN, BM, WN, WM, MODE_1X1>(a, f32, splits, stages, st);
  else if (mode == MODE_TILED)
    launch_mode<BN, BM, WN, WM, MODE_TILED>(a, f32, splits, stages, st);
  else
    launch_mode<BN, BM, WN, WM, MODE_GENERIC>(a, f32, splits, stages, st);
}

// Checks a convolution's shape and fills the launch arguments it implies
// (everything but the pointers).
static dstack_status conv_shape(int N, int H, int W, int C, int K, int R, int S, int stride, int pad, int act,
                                int n_cu, ConvArgs* a) {
  DS_CHECK(C % 8 == 0, DSTACK_E_UNSUPPORTED, "conv2d: C must be a multiple of 8");
  DS_CHECK(K % 4 == 0, DSTACK_E_UNSUPPORTED, "conv2d: K must be a multiple of 4");
  DS_CHECK(N > 0 && H > 0 && W > 0 && K > 0 && R > 0 && S > 0 && stride > 0 && pad >= 0, DSTACK_E_INVALID,
           "conv2d: bad shape");
  DS_CHECK(act >= ACT_NONE && act <= ACT_TANH, DSTACK_E_INVALID, "conv2d: act must be 0..4");
  a->N = N; a->H = H; a->W = W; a->C = C; a->K = K; a->R = R; a->S = S; a->stride = stride; a->pad = pad;
  a->Ho = out_dim(H, R, stride, pad);
  a->Wo = out_dim(W, S, stride, pad);
  DS_CHECK(a->Ho > 0 && a->Wo > 0, DSTACK_E_INVALID, "conv2d: empty output");
  // buffer offsets are 32-bit with bit 31 reserved as the out-of-range marker
  DS_CHECK((long)N * H * W * C * 2 < (1L << 31) && (long)N * a->Ho * a->Wo * K < (1L << 31) &&
               (long)K * R * S * C * 2 < (1L << 31),
           DSTACK_E_UNSUPPORTED, "conv2d: tensor too large for 31-bit byte offsets");
  a->M = N * a->Ho * a->Wo;
  a->Kg = R * S * C;
  a->act = act;
  a->n_cu = n_cu <= 0 ? 256 : n_cu;  // unknown: plan for the whole device
  return DSTACK_OK;
}

// The launch a convolution gets: the streaming 1x1 kernel, or the tiled
// kernel with its tile, split and ring depth.  Split-K is considered only
// with a workspace and arrival counters, and not for an fp32 output (the
// fused reduction stores bf16).
static ConvLaunchPlan conv_launch_plan(const ConvArgs& a, bool out_fp32, bool can_split, size_t split_bytes) {
  ConvLaunchPlan L{};
  const bool one = a.R == 1 && a.S == 1 && a.pad == 0;
  if (one && a.stride == 1 && a.C <= 32 && a.K % 16 == 0 && a.act <= ACT_RELU6) {  // small depth: streaming
    L.kernel = 1;
    int nb = 8;
    while ((a.K / 16) % nb) --nb;
    L.bn = 16 * nb;
    L.mode = MODE_1X1S1;
    L.splits = 1;
    return L;
  }
  L.kernel = 0;
  L.mode = one ? (a.stride == 1 ? MODE_1X1S1 : MODE_1X1) : (a.C % BK == 0 && a.R * a.S <= 32 ? MODE_TILED : MODE_GENERIC);
  const ConvPlan p = choose_plan(a.M, a.K, a.Kg, a.n_cu, can_split && !out_fp32, split_bytes);
  const int nkt = ceil_div(a.Kg, BK);
  L.kt_per_split = ceil_div(nkt, p.splits);
  L.splits = ceil_div(nkt, L.kt_per_split);  // no empty slices
  L.bn = p.bn;
  L.bm = p.bm;
  const long tiles = (long)ceil_div(a.M, p.bm) * ceil_div(a.K, p.bn);
  L.stages = conv_stages(p.bn, p.bm);
  if (L.stages > 2 && short_ring(L.kt_per_split, L.splits, tiles * L.splits, a.n_cu)) L.stages = 2;
  return L;
}

dstack_status conv2d_plan(int N, int H, int W, int C, int K, int R, int S, int stride, int pad, int act,
                          bool out_fp32, int n_cu, size_t split_bytes, ConvLaunchPlan* out) {
  ConvArgs a{};
  dstack_status s = conv_shape(N, H, W, C, K, R, S, stride, pad, act, n_cu, &a);
  if (s != DSTACK_OK) return s;
  *out = conv_launch_plan(a, out_fp32, true, split_bytes);
  out->split_bytes = out->splits > 1 ? (size_t)out->splits * a.M * a.K * sizeof(float) : 0;
  return DSTACK_OK;
}

dstack_status launch_conv2d_ws(const bf16* x, int N, int H, int W, int C, const bf16* w, int K, int R, int S,
                               int stride, int pad, const float* scale, const float* shift, const bf16* res,
                               int act, void* y, bool out_fp32, int n_cu, float* splitk_ws, size_t splitk_bytes,
                               unsigned* tile_counters, hipStream_t st) {
  ConvArgs a{};
  dstack_status s = conv_shape(N, H, W, C, K, R, S, stride, pad, act, n_cu, &a);
  if (s != DSTACK_OK) return s;
  a.x = x; a.w = w; a.scale = scale; a.shift = shift; a.res = res; a.y = y; a.partial = nullptr;
  a.counters = nullptr;
  a.div_wo = FastDiv::make(a.Wo);
  a.div_ho = FastDiv::make(a.Ho);
  a.div_c = FastDiv::make(C);
  a.div_s = FastDiv::make(S);
  const ConvLaunchPlan p =
      conv_launch_plan(a, out_fp32, splitk_ws != nullptr && tile_counters != nullptr, splitk_bytes);
  if (p.kernel == 1) {
    launch_1x1s(a, out_fp32, a.n_cu, st);
    DS_HIP(hipGetLastError());
    return DSTACK_OK;
  }
  a.kt_per_split = p.kt_per_split;
  if (p.splits > 1) {
    a.partial = splitk_ws;
    a.counters = tile_counters;
  }
  if (p.bn == 128 && p.bm == 128)
    launch_cfg<128, 128, 2, 2>(a, p.mode, out_fp32, p.splits, p.stages, st);
  else if (p.bn == 128 && p.bm == 64)
    launch_cfg<128, 64, 2, 2>(a, p.mode, out_fp32, p.splits, p.stages, st);
  else if (p.bn == 64 && p.bm == 128)
    launch_cfg<64, 128, 2, 2>(a, p.mode, out_fp32, p.splits, p.stages, st);
  else if (p.bn == 64 && p.bm == 64)
    launch_cfg<64, 64, 2, 2>(a, p.mode, out_fp32, p.splits, p.stages, st);
  else
    launch_cfg<32, 128, 1, 4>(a, p.mode, out_fp32, p.splits, p.stages, st);
  DS_HIP(hipGetLastError());
  return DSTACK_OK;
}

// ---- the allocation-free variant: split-K scratch in a file-scope array ----
//
// Layout as the caller's workspace of launch_conv2d_ws: the arrival counters
// first, then the fp32 slices.  Every device the library runs on holds its
// own copy until the process ends; host code reaches it only through the
// address hipGetSymbolAddress returns for the current device (the array's
// name is a host-side stand-in, not a device address).
static __device__ __align__(256) unsigned char scratch[CONV_SCRATCH_BYTES];

__global__ __launch_bounds__(256) void zero_words_kernel(unsigned* p, int n) {
  for (int i = blockIdx.x * 256 + threadIdx.x; i < n; i += gridDim.x * 256) p[i] = 0u;
}

constexpr int kMaxDevices = 64;

// The scratch's device address on the current device, looked up once per
// device; at that first lookup its counters are cleared with a fill kernel on
// `st` (no memset node: the call may be under graph capture).
static dstack_status scratch_address(hipStream_t st, unsigned char** out) {
  static std::mutex mu;
  static unsigned char* addr[kMaxDevices] = {};
  int dev = 0;
  DS_HIP(hipGetDevice(&dev));
  DS_CHECK(dev >= 0 && dev < kMaxDevices, DSTACK_E_UNSUPPORTED, "conv2d_noalloc: device index above 63");
  std::lock_guard<std::mutex> g(mu);
  if (!addr[dev]) {
    void* p = nullptr;
    DS_HIP(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    DS_CHECK(p != nullptr && ((uintptr_t)p % 256) == 0, DSTACK_E_HIP, "conv2d_noalloc: no scratch address");
    launch(zero_words_kernel, dim3(SPLITK_TILE_COUNTERS / 256), dim3(256), 0, st, static_cast<unsigned*>(p),
           SPLITK_TILE_COUNTERS);
    DS_HIP(hipGetLastError());
    addr[dev] = static_cast<unsigned char*>(p);
  }
  *out = addr[dev];
  return DSTACK_OK;
}

dstack_status launch_conv2d_noalloc(const bf16* x, int N, int H, int W, int C, const bf16* w, int K, int R, int S,
                                    int stride, int pad, const float* scale, const float* shift, const bf16* res,
                                    int act, void* y, bool out_fp32, int n_cu, hipStream_t st) {
  ConvLaunchPlan p;
  dstack_status s = conv2d_plan(N, H, W, C, K, R, S, stride, pad, act, out_fp32, n_cu, (size_t)1 << 40, &p);
  if (s != DSTACK_OK) return s;
  const size_t counters = SPLITK_TILE_COUNTERS * sizeof(unsigned);
  DS_CHECK(counters + p.split_bytes <= CONV_SCRATCH_BYTES, DSTACK_E_UNSUPPORTED,
           "conv2d_noalloc: this shape's split-K plan needs " + std::to_string(counters + p.split_bytes) +
               " bytes of scratch, above the fixed " + std::to_string(CONV_SCRATCH_BYTES));
  unsigned char* sc = nullptr;
  s = scratch_address(st, &sc);
  if (s != DSTACK_OK) return s;
  return launch_conv2d_ws(x, N, H, W, C, w, K, R, S, stride, pad, scale, shift, res, act, y, out_fp32, n_cu,
                          reinterpret_cast<float*>(sc + counters), CONV_SCRATCH_BYTES - counters,
                          reinterpret_cast<unsigned*>(sc), st);
}

dstack_status launch_conv2d(const bf16* x, int N, int H, int W, int C, const bf16* w, int K, int R, int S,
                            int stride, int pad, const float* scale, const float* shift, const bf16* res, int act,
                            void* y, bool out_fp32, int n_cu, hipStream_t st) {
  return launch_conv2d_ws(x, N, H, W, C, w, K, R, S, stride, pad, scale, shift, res, act, y, out_fp32, n_cu,
                          nullptr, 0, nullptr, st);
}

}  // namespace dstack
