// Shared definitions of the HIP library: bf16 vector types, status and
// error-text plumbing, launch helpers.
#pragma once
#include <hip/hip_runtime.h>

#include <cstdint>
#include <cstdio>
#include <string>
#include <vector>

#include "../../include/dstack.h"

namespace dstack {

// Division by a runtime constant d >= 1 for 0 <= n < 2^31 with a multiply-high:
// l = ceil(log2 d), m = floor(2^32 (2^l - d) / d) + 1, n / d = (mulhi(m, n) + n) >> l
// (Granlund & Montgomery, "Division by invariant integers using
// multiplication", PLDI 1994).
struct FastDiv {
  unsigned m;
  int l;
  int d;
  static FastDiv make(int d) {
    FastDiv f;
    f.d = d;
    f.l = 0;
    while ((1LL << f.l) < d) ++f.l;
    f.m = (unsigned)((((1ULL << 32) * ((1ULL << f.l) - (unsigned long long)d)) / (unsigned long long)d) + 1);
    return f;
  }
  __device__ __forceinline__ int div(int n) const { return (int)((__umulhi(m, (unsigned)n) + (unsigned)n) >> l); }
};

typedef __bf16 bf16;
typedef __attribute__((__vector_size__(8 * sizeof(__bf16)))) __bf16 bf16x8;
typedef __attribute__((__vector_size__(4 * sizeof(__bf16)))) __bf16 bf16x4;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float f32x4;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;

enum Act { ACT_NONE = 0, ACT_RELU = 1, ACT_RELU6 = 2, ACT_GELU = 3, ACT_TANH = 4 };

// Thread-local error text behind dstack_last_error().
void set_error(const std::string& msg);
void clear_error();

// Optional events that a launcher attaches to its kernels' own dispatch
// packets (hipExtLaunchKernelGGL): `start` takes the begin timestamp of the
// first kernel of the operation, `stop` the end timestamp of the last one.
// Set by the per-kernel profiler for one launch at a time; null otherwise.
struct DispatchEvents {
  hipEvent_t start = nullptr, stop = nullptr;
};
DispatchEvents& dispatch_events();

// Launch-shape recording, for the analytical model's per-kernel parallelism:
// while a recorder is installed on the calling thread, launch() notes each
// kernel's workgroup count and how many of its workgroups one CU holds at
// once, and does not launch it.  Every kernel of the library goes through
// launch().
struct LaunchShape {
  long workgroups;
  int per_cu;
};
std::vector<LaunchShape>*& shape_recorder();

template <typename... KArgs, typename... Args>
inline void launch(void (*kernel)(KArgs...), dim3 grid, dim3 block, size_t shmem, hipStream_t st, Args... args) {
  if (std::vector<LaunchShape>* rec = shape_recorder()) {
    int per_cu = 0;
    if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, (int)(block.x * block.y * block.z), shmem) !=
        hipSuccess)
      per_cu = 0;
    rec->push_back(LaunchShape{(long)grid.x * grid.y * grid.z, per_cu});
    return;
  }
  hipLaunchKernelGGL(kernel, grid, block, shmem, st, args...);
}

// Analytical DNN model (Sec. 4.3); the C ABI wraps these.
dstack_status knee_model_sequence(int p, int b, int kmax, double* n_out);
dstack_status knee_model_eval(const dstack_knee_model* km, const int* s_values, int n_s, double* et_out,
                              int* knee_index);

inline dstack_status fail(dstack_status st, const std::string& msg) {
  set_error(msg);
  return st;
}

inline dstack_status hip_fail(hipError_t e, const char* what) {
  return fail(DSTACK_E_HIP, std::string(what) + ": " + hipGetErrorString(e));
}

#define DS_HIP(call)                                        \
  do {                                                      \
    hipError_t e_ = (call);                                 \
    if (e_ != hipSuccess) return ::dstack::hip_fail(e_, #call); \
  } while (0)

#define DS_CHECK(cond, st, msg)                      \
  do {                                               \
    if (!(cond)) return ::dstack::fail((st), (msg)); \
  } while (0)

inline int ceil_div(int a, int b) { return (a + b - 1) / b; }
inline int out_dim(int in, int k, int stride, int pad) { return (in + 2 * pad - k) / stride + 1; }

// GELU with the Gaussian CDF through erf (the transformer's activation)
__device__ __forceinline__ float gelu_erf(float v) { return 0.5f * v * (1.0f + erff(v * 0.70710678118654752f)); }

__device__ __forceinline__ float apply_act(float v, int act) {
  if (act == ACT_RELU) return fmaxf(v, 0.0f);
  if (act == ACT_RELU6) return fminf(fmaxf(v, 0.0f), 6.0f);
  if (act == ACT_GELU) return gelu_erf(v);
  if (act == ACT_TANH) return tanhf(v);
  return v;
}

// split-K arrival counters per model workspace (conv tiles of one launch)
constexpr int SPLITK_TILE_COUNTERS = 4096;

// The launch a convolution gets: kernel 0 = the tiled implicit GEMM (tile
// bn x bm, split-K slices of kt_per_split depth tiles, an LDS ring of
// `stages` tiles, activation addressing `mode`), 1 = the streaming 1x1
// kernel of small depth (bn = channels per wave); split_bytes = fp32 slice
// bytes of a split plan (0 without a split).
struct ConvLaunchPlan {
  int kernel, mode, bn, bm, splits, kt_per_split, stages;
  size_t split_bytes;
};
// Host only: the plan launch_conv2d_ws would take on n_cu CUs with
// split_bytes of slice workspace (and arrival counters).
dstack_status conv2d_plan(int N, int H, int W, int C, int K, int R, int S, int stride, int pad, int act,
                          bool out_fp32, int n_cu, size_t split_bytes, ConvLaunchPlan* out);
// Fixed split-K scratch of the allocation-free convolution: 16 KiB of
// arrival counters plus 32 MiB of slices, per device.
constexpr size_t CONV_SCRATCH_BYTES = SPLITK_TILE_COUNTERS * sizeof(unsigned) + ((size_t)32 << 20);
// launch_conv2d_ws with the library's fixed scratch in place of a workspace
// (the plan it would take with an unlimited one; E_UNSUPPORTED if that plan
// needs more than CONV_SCRATCH_BYTES).  Allocates nothing.
dstack_status launch_conv2d_noalloc(const bf16* x, int N, int H, int W, int C, const bf16* w, int K, int R, int S,
                                    int stride, int pad, const float* scale, const float* shift, const bf16* res,
                                    int act, void* y, bool out_fp32, int n_cu, hipStream_t st);

// ---- kernel launchers (defined in the .hip files) ----
dstack_status launch_conv2d(const bf16* x, int N, int H, int W, int C, const bf16* w, int K, int R, int S,
                            int stride, int pad, const float* scale, const float* shift, const bf16* res, int act,
                            void* y, bool out_fp32, int n_cu, hipStream_t st);
dstack_status launch_dwconv3x3(const bf16* x, int N, int H, int W, int C, const bf16* w_rsc, int stride,
                               const float* scale, const float* shift, int act, bf16* y, hipStream_t st);
// ws: fp32 partial sums of a depth split (fc_workspace_bytes for n_cu CUs);
// NULL or too small runs fewer splits.  packed: w in MFMA fragment order
// (as a model packs its FC weights at load), else row-major [O][I].
size_t fc_workspace_bytes(int B, int I, int O, int n_cu);
dstack_status launch_fc(const bf16* x, int B, int I, const bf16* w, const float* bias, int O, int act, void* y,
                        bool out_fp32, int n_cu, float* ws, size_t ws_bytes, hipStream_t st, bool packed = false);
dstack_status launch_maxpool(const bf16* x, int N, int H, int W, int C, int k, int stride, int pad, bf16* y,
                             hipStream_t st);
dstack_status launch_avgpool(const bf16* x, int N, int H, int W, int C, bf16* y, hipStream_t st);
dstack_status launch_expand_dw(const bf16* x, int N, int H, int W, int Cin, const bf16* we, int Ce, const float* se,
                               const float* he, int act_e, const bf16* wd, int stride, const float* sd,
                               const float* hd, int act_d, bf16* y, hipStream_t st);
dstack_status launch_embed_ln(const int* ids, int rows, int T, int vocab, const bf16* we, const bf16* pe,
                              const bf16* te, int H, const float* gamma, const float* beta, float eps, bf16* y,
                              hipStream_t st);
dstack_status launch_layernorm(const bf16* x, int rows, int H, const float* gamma, const float* beta, float eps,
                               bf16* y, hipStream_t st);
dstack_status launch_attention(const bf16* qkv, int B, int T, int heads, int dh, bf16* out, hipStream_t st);
dstack_status launch_conv2d_rgb(const bf16* x, int N, int H, int W, const bf16* w4, int K, int R, int stride, int pad,
                                const float* scale, const float* shift, int act, bf16* y, hipStream_t st);
dstack_status launch_lstm_pack_whh(const bf16* w_hh, bf16* wp, int H, hipStream_t st);
dstack_status launch_lstm_step(const float* gx_t, const bf16* wp, const bf16* hp_prev, float* c, bf16* h_next,
                               bf16* hp_next, float* h_f32, int B, int H, bool first, int n_cu, hipStream_t st);
int lstm_units_per_block(int B, int H, int n_cu);
dstack_status launch_probe(uint32_t* d_out, int n_blocks, hipStream_t st);

}  // namespace dstack
