// Model builder and executor: the five architectures as flat lists of
// kernel launches over NHWC bf16 activations, with per-(model, partition)
// workspaces.
#pragma once
#include <atomic>
#include <map>
#include <memory>
#include <mutex>
#include <string>
#include <vector>

#include "common.hpp"

namespace dstack {

enum Dist { DIST_HE = 0, DIST_ZERO = 1, DIST_LSTM = 2 };

struct TensorSpec {
  int64_t numel = 0;
  int dist = DIST_HE;
  int fan_in = 0;
  // device placement
  int64_t dev_off = 0;   // bf16 elements into the weight arena
  int layout = 0;        // 0 same as logical, 1 conv stem padded C->8, 2 depthwise [C][3][3] -> [3][3][C],
                         // 3 RGB stem padded C->4
  int d0 = 0, d1 = 0, d2 = 0, d3 = 0;  // logical dims for re-layout
};
// elements of a tensor's device layout
inline int64_t dev_numel(const TensorSpec& t) {
  if (t.layout == 1) return (int64_t)t.d0 * t.d1 * t.d2 * 8;
  if (t.layout == 3) return (int64_t)t.d0 * t.d1 * t.d2 * 4;
  return t.numel;
}


uint16_t bf16_from_double(double x);
void generate_tensor(uint64_t seed, int index, const TensorSpec& t, uint16_t* out);

enum OpKind { OP_CONV, OP_DW, OP_MAXPOOL, OP_AVGPOOL, OP_FC, OP_LSTM, OP_CONV_RGB, OP_EXPAND_DW, OP_EMBED_LN,
              OP_LAYERNORM, OP_ATTENTION };
enum KernelClass { KC_MFMA = 0, KC_DW = 1, KC_FC = 2, KC_LSTM = 3, KC_GLUE = 4, KC_DIRECT = 5, KC_EXPAND_DW = 6,
                   KC_ATTENTION = 7 };

constexpr int BUF_IN = -1;
constexpr int BUF_OUT = -2;
constexpr int BUF_NONE = -3;

struct Op {
  OpKind kind;
  int in = BUF_NONE, out = BUF_NONE, res = BUF_NONE;
  int H = 0, W = 0, C = 0, K = 0, R = 1, S = 1, stride = 1, pad = 0, act = 0, Ho = 0, Wo = 0;
  int C_true = 0;           // channels before padding (FLOP accounting)
  int64_t w_off = 0;        // bf16 elements into the weight arena
  int64_t scale_off = -1;   // fp32 elements into the fp32 arena (-1: none)
  int64_t shift_off = -1;
  int out_f32 = 0;
  // fused expand + depthwise: the depthwise weights, BN and activation;
  // token embedding: position (w2_off) and token-type (w3_off) tables
  int64_t w2_off = 0, scale2_off = -1, shift2_off = -1, w3_off = 0;
  int act2 = 0;
  // LSTM layer
  int T = 0, I = 0, Hd = 0;
  int64_t wih_off = 0, whh_off = 0, bias_off = 0;
  // FC weights / LSTM W_hh in MFMA fragment order: elements into the packed arena (-1: none)
  int64_t wp_off = -1;
  // tensor indices used when folding biases / BN at upload (-1: none)
  int w_t = -1, bias_t = -1, bn = 0;
  int wih_t = -1, whh_t = -1, bih_t = -1, bhh_t = -1;
};

struct KernelTimer;  // optional per-kernel event recorder

struct Workspace {
  void* base = nullptr;
  size_t bytes = 0;
  std::vector<char*> bufs;
  float* splitk = nullptr;
  size_t splitk_bytes = 0;
  unsigned* tile_counters = nullptr;  // SPLITK_TILE_COUNTERS split-K arrival counters, zero between launches
  float* lstm_gx = nullptr;
  float* lstm_c = nullptr;
  bf16* lstm_h[2] = {nullptr, nullptr};
  bf16* lstm_hp = nullptr;  // h(t-1), h(t) in fragment order (2 x max batch x H)
  std::atomic<bool> busy{false};
  // captured forward passes, keyed by (batch, input, output, CUs of the
  // partition); replayed with one hipGraphLaunch
  struct GraphKey {
    int batch;
    const void* in;
    void* out;
    int n_cu;
    bool operator<(const GraphKey& o) const {
      if (batch != o.batch) return batch < o.batch;
      if (in != o.in) return in < o.in;
      if (out != o.out) return out < o.out;
      return n_cu < o.n_cu;
    }
  };
  std::map<GraphKey, hipGraphExec_t> graphs;
  std::vector<GraphKey> graph_order;  // insertion order, for eviction
  ~Workspace();
};

struct Model {
  std::string arch;
  uint64_t seed = 0;
  int is_lstm = 0;
  int max_batch = 32;
  int in_h = 0, in_w = 0, in_c = 0;
  int seq_len = 0, in_features = 0, out_features = 0;
  int input_tokens = 0;  // 1: the input is int32 token ids [batch][seq_len]
  std::vector<TensorSpec> tensors;
  std::vector<Op> ops;
  std::vector<int64_t> buf_elems;   // per-item bf16 elements of each buffer id
  int64_t n_weights = 0;            // bf16 arena size
  int64_t n_fp32 = 0;               // fp32 arena size
  std::vector<float> fp32_host;     // scale/shift/bias values
  bf16* d_w = nullptr;
  float* d_f32 = nullptr;
  bf16* d_wp = nullptr;             // packed copies of the weight-streaming operands
  int64_t n_wp = 0;
  int lstm_T = 0, lstm_B_max = 32, lstm_H = 0;
  std::mutex ws_mu;
  std::map<int, std::unique_ptr<Workspace>> ws;  // by partition id
  // scratch for knee sweeps
  void* sweep_in = nullptr;
  void* sweep_out = nullptr;

  ~Model();
};

// Architecture description (host only; no device memory touched).
dstack_status build_arch(const std::string& arch, Model& m);
// Device upload of the generated weights and folded BN parameters.
dstack_status upload_weights(Model& m);
// Workspace for batch <= max_batch, on demand.
dstack_status get_workspace(Model& m, int partition_id, int n_cu, hipStream_t st, Workspace** out);
// Frees the workspace (and its captured graphs) kept for a partition id, if
// any and not in use; called when the partition is destroyed.
void release_workspace(Model& m, int partition_id);

// Enqueue one forward pass on `st`.  `timer` may be null.  n_ops >= 0 runs
// only the first n_ops ops; last_out (may be null) receives the output
// buffer of the last op run.
dstack_status forward(Model& m, int batch, const void* d_in, void* d_out, Workspace& ws, int n_cu, hipStream_t st,
                      KernelTimer* timer, int n_ops = -1, void** last_out = nullptr);

// Algorithmic cost of the ops at a batch size.
void model_cost(const Model& m, int batch, double* flops, double* mfma_flops, double* weight_bytes, int* n_kernels);

struct KernelTimer {
  struct Rec {
    int kind;
    double flops, bytes;
    hipEvent_t a, b;
    int m, n, k;
  };
  hipStream_t st;
  std::vector<Rec> recs;
  hipEvent_t pending = nullptr;
  hipEvent_t ds_start = nullptr, ds_stop = nullptr;  // armed dispatch events (before_dispatch)
  // dry mode: no events; each timed unit notes the range of launch shapes
  // the installed recorder took for it
  bool dry = false;
  struct Unit {
    int kind;
    size_t l0, l1;
    double flops, bytes;
  };
  std::vector<Unit> units;
  size_t unit_l0 = 0;
  void before();
  void before_dispatch();
  void after(int kind, double flops, double bytes, int m = 0, int n = 0, int k = 0);
  ~KernelTimer();
};

size_t conv_splitk_workspace_bytes(int M, int K, int Kg, int n_cu);
dstack_status launch_conv2d_ws(const bf16* x, int N, int H, int W, int C, const bf16* w, int K, int R, int S,
                               int stride, int pad, const float* scale, const float* shift, const bf16* res,
                               int act, void* y, bool out_fp32, int n_cu, float* splitk_ws, size_t splitk_bytes,
                               unsigned* tile_counters, hipStream_t st);
// whh_packed: W_hh already in fragment order (a model's, packed at load), or
// NULL: w_hh is packed into wp_scratch (4H x H) first.
dstack_status lstm_layer_run(const bf16* x, int T, int B, int I, int H, const bf16* w_ih, const bf16* w_hh,
                             const bf16* whh_packed, const float* bias, bf16* h_bf16, float* h_f32, float* gx,
                             float* c, bf16* wp_scratch, bf16* hp, int n_cu, hipStream_t st, KernelTimer* timer);

}  // namespace dstack
