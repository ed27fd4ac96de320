// C ABI of the library: partitions (CU-masked streams), models, inference,
// knee sweep, scheduling and kernel-level entry points.  Every function
// catches C++ exceptions and converts them to a status.
#include <hip/hip_ext.h>

#include <algorithm>
#include <chrono>
#include <atomic>
#include <cmath>
#include <cstdlib>
#include <cstdint>
#include <cstring>
#include <mutex>
#include <new>
#include <set>
#include <string>
#include <vector>

#include "launcher.hpp"
#include "model.hpp"
#include "sched.hpp"

using namespace dstack;

namespace dstack {

static thread_local std::string t_err;
void set_error(const std::string& msg) { t_err = msg; }
void clear_error() { t_err.clear(); }

}  // namespace dstack

struct dstack_partition_s {
  int id;
  uint32_t slot_mask;
  int n_slots;
  int n_cu;
  uint32_t words[8];
  hipStream_t stream;
};

struct dstack_model_s {
  Model m;
};

namespace {

// Partition ids start at 16: workspace ids below that are the library's own
// (knee sweeps 0, GPU% change probes 1 and 2, the live launcher's models 4..7),
// never a partition's.
std::atomic<int> g_next_partition_id{16};

// Live partitions.  Each owns one CU-masked HIP stream, and a CU-masked
// stream gets a hardware queue of its own.  A run with five live masked
// streams (four of them busy) beside one unmasked stream stopped making
// progress, while runs with up to four live masked streams (all of them busy
// at once) completed; the cause is not known, so a fifth live partition is
// refused before its stream is created.
constexpr int kMaxLivePartitions = 4;
std::mutex g_part_mu;
int g_live_partitions = 0;

// Loaded models, so that destroying a partition can release the workspaces
// (activations, split-K slices, captured graphs) each model holds for it.
std::mutex g_model_mu;
std::set<dstack_model_s*> g_models;

template <typename F>
dstack_status guarded(F&& f) {
  try {
    clear_error();
    return f();
  } catch (const std::bad_alloc&) {
    return fail(DSTACK_E_OOM, "host allocation failed");
  } catch (const std::exception& e) {
    return fail(DSTACK_E_STATE, std::string("internal error: ") + e.what());
  } catch (...) {
    return fail(DSTACK_E_STATE, "internal error");
  }
}

dstack_status make_partition(uint32_t slot_mask, dstack_partition* out) {
  DS_CHECK(out, DSTACK_E_INVALID, "partition: null out pointer");
  DS_CHECK(slot_mask != 0, DSTACK_E_INVALID, "partition: empty slot set");
  {
    std::lock_guard<std::mutex> g(g_part_mu);
    DS_CHECK(g_live_partitions < kMaxLivePartitions, DSTACK_E_UNSUPPORTED,
             "partition: at most " + std::to_string(kMaxLivePartitions) +
                 " live partitions (CU-masked streams); destroy one first");
    ++g_live_partitions;  // reserved before the stream exists
  }
  auto unreserve = [] {
    std::lock_guard<std::mutex> g(g_part_mu);
    --g_live_partitions;
  };
  auto* p = new (std::nothrow) dstack_partition_s();
  if (!p) {
    unreserve();
    return fail(DSTACK_E_OOM, "partition: host allocation failed");
  }
  p->id = g_next_partition_id++;
  p->slot_mask = slot_mask;
  p->n_slots = __builtin_popcount(slot_mask);
  p->n_cu = p->n_slots * DSTACK_CUS_PER_SLOT;
  std::memset(p->words, 0, sizeof(p->words));
  // slot j = mask bits 8j..8j+7 = CU j of each of the 8 XCDs (bit i -> XCD i % 8)
  for (int j = 0; j < DSTACK_TOTAL_SLOTS; ++j)
    if ((slot_mask >> j) & 1) p->words[j / 4] |= 0xFFu << (8 * (j % 4));
  hipError_t e = hipExtStreamCreateWithCUMask(&p->stream, 8, p->words);
  if (e != hipSuccess) {
    delete p;
    unreserve();
    return hip_fail(e, "hipExtStreamCreateWithCUMask");
  }
  *out = p;
  return DSTACK_OK;
}

dstack_status slots_from_fraction(double f, int* slots) {
  DS_CHECK(slots, DSTACK_E_INVALID, "fraction: null out pointer");
  DS_CHECK(std::isfinite(f) && f > 0.0 && f <= 1.0, DSTACK_E_INVALID, "fraction must be in (0, 1]");
  int s = (int)std::floor(32.0 * f + 0.5);
  *slots = std::min(32, std::max(1, s));
  return DSTACK_OK;
}

}  // namespace

extern "C" {

const char* dstack_last_error(void) { return t_err.c_str(); }

dstack_status dstack_fraction_to_slots(double f, int* slots) {
  return guarded([&] { return slots_from_fraction(f, slots); });
}

dstack_status dstack_partition_create(double f, dstack_partition* out) {
  return guarded([&] {
    int s;
    dstack_status st = slots_from_fraction(f, &s);
    if (st != DSTACK_OK) return st;
    return make_partition(s == 32 ? 0xFFFFFFFFu : ((1u << s) - 1), out);
  });
}

dstack_status dstack_partition_create_at(int off, int n, dstack_partition* out) {
  return guarded([&] {
    DS_CHECK(off >= 0 && n >= 1 && off + n <= DSTACK_TOTAL_SLOTS, DSTACK_E_INVALID, "slot range outside 0..32");
    uint32_t m = (n == 32) ? 0xFFFFFFFFu : (((1u << n) - 1) << off);
    return make_partition(m, out);
  });
}

dstack_status dstack_partition_create_mask(uint32_t slot_mask, dstack_partition* out) {
  return guarded([&] { return make_partition(slot_mask, out); });
}

dstack_status dstack_partition_query(dstack_partition p, int* n_cu, uint32_t mask_words[8], void** hip_stream) {
  return guarded([&] {
    DS_CHECK(p, DSTACK_E_INVALID, "null partition");
    if (n_cu) *n_cu = p->n_cu;
    if (mask_words) std::memcpy(mask_words, p->words, sizeof(p->words));
    if (hip_stream) *hip_stream = (void*)p->stream;
    return DSTACK_OK;
  });
}

dstack_status dstack_synchronize(dstack_partition p) {
  return guarded([&] {
    DS_CHECK(p, DSTACK_E_INVALID, "null partition");
    DS_HIP(hipStreamSynchronize(p->stream));
    return DSTACK_OK;
  });
}

dstack_status dstack_partition_count(int* live, int* max_live) {
  return guarded([&] {
    std::lock_guard<std::mutex> g(g_part_mu);
    if (live) *live = g_live_partitions;
    if (max_live) *max_live = kMaxLivePartitions;
    return DSTACK_OK;
  });
}

void dstack_partition_destroy(dstack_partition p) {
  if (!p) return;
  (void)hipStreamSynchronize(p->stream);
  {
    std::lock_guard<std::mutex> g(g_model_mu);
    for (dstack_model_s* h : g_models) release_workspace(h->m, p->id);
  }
  (void)hipStreamDestroy(p->stream);
  delete p;
  std::lock_guard<std::mutex> g(g_part_mu);
  --g_live_partitions;
}

dstack_status dstack_probe_cu_ids(dstack_partition p, int n_blocks, int via_graph, uint32_t* host_out) {
  return guarded([&] {
    DS_CHECK(p && host_out, DSTACK_E_INVALID, "probe: null pointer");
    DS_CHECK(n_blocks >= 1 && n_blocks <= 65536, DSTACK_E_INVALID, "probe: n_blocks in 1..65536");
    uint32_t* d = nullptr;
    DS_HIP(hipMalloc(&d, (size_t)n_blocks * 8));
    dstack_status s = DSTACK_OK;
    hipError_t e = hipSuccess;
    if (via_graph) {
      hipGraph_t g = nullptr;
      hipGraphExec_t ex = nullptr;
      e = hipStreamBeginCapture(p->stream, hipStreamCaptureModeThreadLocal);
      if (e == hipSuccess) {
        s = launch_probe(d, n_blocks, p->stream);
        e = hipStreamEndCapture(p->stream, &g);
      }
      if (s == DSTACK_OK && e == hipSuccess) e = hipGraphInstantiate(&ex, g, nullptr, nullptr, 0);
      if (s == DSTACK_OK && e == hipSuccess) e = hipGraphLaunch(ex, p->stream);
      if (e == hipSuccess && s == DSTACK_OK) e = hipStreamSynchronize(p->stream);
      if (ex) (void)hipGraphExecDestroy(ex);
      if (g) (void)hipGraphDestroy(g);
    } else {
      s = launch_probe(d, n_blocks, p->stream);
    }
    if (s == DSTACK_OK && e == hipSuccess) e = hipStreamSynchronize(p->stream);
    if (s == DSTACK_OK && e == hipSuccess) e = hipMemcpy(host_out, d, (size_t)n_blocks * 8, hipMemcpyDeviceToHost);
    (void)hipFree(d);
    if (s != DSTACK_OK) return s;
    if (e != hipSuccess) return hip_fail(e, "probe");
    return DSTACK_OK;
  });
}

dstack_status dstack_model_load(const char* arch, uint64_t seed, dstack_model* out) {
  return guarded([&] {
    DS_CHECK(arch && out, DSTACK_E_INVALID, "model_load: null pointer");
    auto* h = new dstack_model_s();
    h->m.seed = seed;
    dstack_status s = build_arch(arch, h->m);
    if (s == DSTACK_OK) s = upload_weights(h->m);
    if (s != DSTACK_OK) {
      std::string msg = t_err;
      delete h;
      set_error(msg);
      return s;
    }
    {
      std::lock_guard<std::mutex> g(g_model_mu);
      g_models.insert(h);
    }
    *out = h;
    return DSTACK_OK;
  });
}

dstack_status dstack_model_query(dstack_model h, dstack_model_info* out) {
  return guarded([&] {
    DS_CHECK(h && out, DSTACK_E_INVALID, "model_query: null pointer");
    const Model& m = h->m;
    std::memset(out, 0, sizeof(*out));
    std::strncpy(out->arch, m.arch.c_str(), sizeof(out->arch) - 1);
    out->is_lstm = m.is_lstm;
    out->max_batch = m.max_batch;
    out->in_h = m.in_h;
    out->in_w = m.in_w;
    out->in_c = m.in_c;
    out->seq_len = m.seq_len;
    out->in_features = m.in_features;
    out->out_features = m.out_features;
    out->input_tokens = m.input_tokens;
    out->num_tensors = (int)m.tensors.size();
    int64_t np = 0;
    for (const auto& t : m.tensors) np += t.numel;
    out->num_params = np;
    double f, mf, wb;
    int nk;
    model_cost(m, 1, &f, &mf, &wb, &nk);
    out->flops_per_item = f;
    out->mfma_flops_per_item = mf;
    out->weight_bytes = wb;
    out->num_kernels = nk;
    return DSTACK_OK;
  });
}

static void unlayout(const TensorSpec& t, const uint16_t* dev, uint16_t* logical) {
  if (t.layout == 0) {
    std::memcpy(logical, dev, (size_t)t.numel * 2);
  } else if (t.layout == 1) {
    int64_t krs = (int64_t)t.d0 * t.d1 * t.d2;
    for (int64_t q = 0; q < krs; ++q)
      for (int c = 0; c < t.d3; ++c) logical[q * t.d3 + c] = dev[q * 8 + c];
  } else if (t.layout == 3) {
    int64_t krs = (int64_t)t.d0 * t.d1 * t.d2;
    for (int64_t q = 0; q < krs; ++q)
      for (int c = 0; c < t.d3; ++c) logical[q * t.d3 + c] = dev[q * 4 + c];
  } else {
    int C = t.d0;
    for (int c = 0; c < C; ++c)
      for (int rs = 0; rs < 9; ++rs) logical[(size_t)c * 9 + rs] = dev[(size_t)rs * C + c];
  }
}

dstack_status dstack_model_export_params(dstack_model h, int idx, void* dst, size_t bytes) {
  return guarded([&] {
    DS_CHECK(h && dst, DSTACK_E_INVALID, "export: null pointer");
    const Model& m = h->m;
    DS_CHECK(idx >= 0 && idx < (int)m.tensors.size(), DSTACK_E_INVALID, "export: tensor index out of range");
    const TensorSpec& t = m.tensors[idx];
    DS_CHECK(bytes == (size_t)t.numel * 2, DSTACK_E_INVALID, "export: byte count must be 2 * numel");
    const int64_t n_dev = dev_numel(t);
    std::vector<uint16_t> tmp((size_t)n_dev);
    DS_HIP(hipMemcpy(tmp.data(), m.d_w + t.dev_off, (size_t)n_dev * 2, hipMemcpyDeviceToHost));
    unlayout(t, tmp.data(), (uint16_t*)dst);
    return DSTACK_OK;
  });
}

void dstack_model_destroy(dstack_model h) {
  if (!h) return;
  (void)hipDeviceSynchronize();
  {
    std::lock_guard<std::mutex> g(g_model_mu);
    g_models.erase(h);
  }
  delete h;
}

dstack_status dstack_generate_params(const char* arch, uint64_t seed, int idx, void* dst, size_t bytes,
                                     int64_t* numel) {
  return guarded([&] {
    DS_CHECK(arch, DSTACK_E_INVALID, "generate: null arch");
    Model m;
    m.seed = seed;
    dstack_status s = build_arch(arch, m);
    if (s != DSTACK_OK) return s;
    DS_CHECK(idx >= 0 && idx < (int)m.tensors.size(), DSTACK_E_INVALID, "generate: tensor index out of range");
    const TensorSpec& t = m.tensors[idx];
    if (numel) *numel = t.numel;
    if (!dst) return DSTACK_OK;
    DS_CHECK(bytes == (size_t)t.numel * 2, DSTACK_E_INVALID, "generate: byte count must be 2 * numel");
    generate_tensor(seed, idx, t, (uint16_t*)dst);
    return DSTACK_OK;
  });
}

// ---------------------------------------------------------------- infer ----

namespace {

struct BusyGuard {
  std::atomic<bool>& f;
  bool ok;
  explicit BusyGuard(std::atomic<bool>& flag) : f(flag) {
    bool expected = false;
    ok = f.compare_exchange_strong(expected, true);
  }
  ~BusyGuard() {
    if (ok) f.store(false);
  }
};

dstack_status check_batch(const Model& m, int batch) {
  DS_CHECK(batch >= 1 && batch <= m.max_batch, DSTACK_E_INVALID,
           "batch must be in 1.." + std::to_string(m.max_batch));
  return DSTACK_OK;
}

// Workspace id 0 is reserved for knee sweeps, which run one partition at a
// time and reuse a single workspace across fractions.
constexpr int SWEEP_WS_ID = 0;
constexpr size_t kMaxGraphsPerWorkspace = 64;

// Forward passes are replayed as HIP graphs unless DSTACK_GRAPH=0.
bool graphs_enabled() {
  static const bool on = [] {
    const char* v = std::getenv("DSTACK_GRAPH");
    return !(v && v[0] == '0');
  }();
  return on;
}

// capture_n_cu > 0: only record and instantiate the graph of a forward
// planned for that many CUs (on p's stream, which runs nothing), so that a
// later call on a partition of that size finds it.
dstack_status infer_impl(Model& m, int batch, const void* d_in, void* d_out, dstack_partition p, KernelTimer* timer,
                         int ws_id = -1, int capture_n_cu = 0) {
  DS_CHECK(d_in && d_out && p, DSTACK_E_INVALID, "infer: null pointer");
  dstack_status s = check_batch(m, batch);
  if (s != DSTACK_OK) return s;
  Workspace* ws;
  s = get_workspace(m, ws_id >= 0 ? ws_id : p->id, p->n_cu, p->stream, &ws);
  if (s != DSTACK_OK) return s;
  BusyGuard g(ws->busy);
  DS_CHECK(g.ok, DSTACK_E_STATE, "infer: another call on this (model, partition) is in progress");
  if (timer || !graphs_enabled())
    return capture_n_cu > 0 ? DSTACK_OK : forward(m, batch, d_in, d_out, *ws, p->n_cu, p->stream, timer);
  // one forward = one graph launch: captured on first use of this key
  const int n_cu = capture_n_cu > 0 ? capture_n_cu : p->n_cu;
  const Workspace::GraphKey key{batch, d_in, d_out, n_cu};
  auto it = ws->graphs.find(key);
  if (it == ws->graphs.end()) {
    DS_HIP(hipStreamBeginCapture(p->stream, hipStreamCaptureModeThreadLocal));
    s = forward(m, batch, d_in, d_out, *ws, n_cu, p->stream, nullptr);
    hipGraph_t graph = nullptr;
    hipError_t e = hipStreamEndCapture(p->stream, &graph);
    if (s != DSTACK_OK) {
      if (graph) (void)hipGraphDestroy(graph);
      return s;
    }
    if (e != hipSuccess) return hip_fail(e, "hipStreamEndCapture");
    hipGraphExec_t exec = nullptr;
    e = hipGraphInstantiate(&exec, graph, nullptr, nullptr, 0);
    (void)hipGraphDestroy(graph);
    if (e != hipSuccess) return hip_fail(e, "hipGraphInstantiate");
    if (ws->graph_order.size() >= kMaxGraphsPerWorkspace) {  // evict the oldest capture
      auto old = ws->graphs.find(ws->graph_order.front());
      (void)hipGraphExecDestroy(old->second);
      ws->graphs.erase(old);
      ws->graph_order.erase(ws->graph_order.begin());
    }
    it = ws->graphs.emplace(key, exec).first;
    ws->graph_order.push_back(key);
  }
  if (capture_n_cu > 0) return DSTACK_OK;
  DS_HIP(hipGraphLaunch(it->second, p->stream));
  return DSTACK_OK;
}

}  // namespace



dstack_status dstack_infer(dstack_model h, int batch, const void* d_in, void* d_out, dstack_partition p) {
  return guarded([&] {
    DS_CHECK(h, DSTACK_E_INVALID, "infer: null model");
    return infer_impl(h->m, batch, d_in, d_out, p, nullptr);
  });
}

dstack_status dstack_infer_hidden(dstack_model h, int batch, const void* d_in, int layer, void* d_hidden,
                                  dstack_partition p) {
  return guarded([&] {
    DS_CHECK(h && d_in && d_hidden && p, DSTACK_E_INVALID, "infer_hidden: null pointer");
    Model& m = h->m;
    DS_CHECK(m.input_tokens, DSTACK_E_UNSUPPORTED, "infer_hidden: only the transformer models have hidden states");
    dstack_status s = check_batch(m, batch);
    if (s != DSTACK_OK) return s;
    // the op that ends each stage: the embedding (+ layer norm), then every
    // second layer norm (the one closing an encoder layer)
    std::vector<int> ends;
    int n_ln = 0;
    for (size_t i = 0; i < m.ops.size(); ++i) {
      if (m.ops[i].kind == OP_EMBED_LN) ends.push_back((int)i);
      if (m.ops[i].kind == OP_LAYERNORM && ++n_ln % 2 == 0) ends.push_back((int)i);
    }
    const int n_layers = (int)ends.size() - 1;
    if (layer < 0) layer = n_layers;
    DS_CHECK(layer <= n_layers, DSTACK_E_INVALID, "infer_hidden: layer must be in 0.." + std::to_string(n_layers));
    Workspace* ws;
    s = get_workspace(m, p->id, p->n_cu, p->stream, &ws);
    if (s != DSTACK_OK) return s;
    BusyGuard g(ws->busy);
    DS_CHECK(g.ok, DSTACK_E_STATE, "infer_hidden: another call on this (model, partition) is in progress");
    void* hid = nullptr;
    s = forward(m, batch, d_in, nullptr, *ws, p->n_cu, p->stream, nullptr, ends[layer] + 1, &hid);
    if (s != DSTACK_OK) return s;
    const Op& op = m.ops[ends[layer]];
    const size_t bytes = (size_t)batch * (op.kind == OP_EMBED_LN ? (size_t)op.T * op.C : (size_t)op.H * op.W * op.C) * 2;
    DS_HIP(hipMemcpyAsync(d_hidden, hid, bytes, hipMemcpyDeviceToDevice, p->stream));
    return DSTACK_OK;
  });
}

dstack_status dstack_profile_layers(dstack_model h, int batch, const void* d_in, void* d_out, dstack_partition p,
                                    dstack_layer_time* out, int max_layers, int* n_layers) {
  return guarded([&] {
    DS_CHECK(h && out && n_layers && p, DSTACK_E_INVALID, "profile: null pointer");
    KernelTimer timer;
    timer.st = p->stream;
    dstack_status s = infer_impl(h->m, batch, d_in, d_out, p, &timer);
    if (s != DSTACK_OK) return s;
    DS_HIP(hipStreamSynchronize(p->stream));
    int n = 0;
    for (auto& r : timer.recs) {
      if (n >= max_layers) break;
      float ms = 0.f;
      DS_HIP(hipEventElapsedTime(&ms, r.a, r.b));
      out[n++] = dstack_layer_time{r.kind, ms, r.flops, r.bytes, r.m, r.n, r.k};
    }
    *n_layers = n;
    return DSTACK_OK;
  });
}

// ----------------------------------------------------------- knee sweep ----

namespace {

// Scratch input/output of the model at its maximum batch for profiling runs
// (contents: a fixed xorshift pattern of values in about [-1, 1), or of
// token ids for a transformer).
dstack_status ensure_sweep_buffers(Model& m) {
  if (m.sweep_in) return DSTACK_OK;
  size_t in_bytes = m.is_lstm        ? (size_t)m.seq_len * m.max_batch * m.in_features * 2
                    : m.input_tokens ? (size_t)m.seq_len * m.max_batch * 4
                                     : (size_t)m.max_batch * m.in_h * m.in_w * m.in_c * 2;
  size_t out_bytes = m.is_lstm ? (size_t)m.seq_len * m.max_batch * m.out_features * 4
                               : (size_t)m.max_batch * m.out_features * 4;
  DS_HIP(hipMalloc(&m.sweep_in, in_bytes));
  DS_HIP(hipMalloc(&m.sweep_out, out_bytes));
  uint64_t z = 0x2545F4914F6CDD1DULL;
  if (m.input_tokens) {  // token ids below 30000
    std::vector<int32_t> ids(in_bytes / 4);
    for (auto& v : ids) {
      z ^= z << 13; z ^= z >> 7; z ^= z << 17;
      v = (int32_t)(z % 30000);
    }
    DS_HIP(hipMemcpy(m.sweep_in, ids.data(), in_bytes, hipMemcpyHostToDevice));
    return DSTACK_OK;
  }
  std::vector<uint16_t> pat(in_bytes / 2);
  for (auto& v : pat) {
    z ^= z << 13; z ^= z >> 7; z ^= z << 17;
    v = bf16_from_double(((double)(z >> 11) * (1.0 / 9007199254740992.0)) * 2.0 - 1.0);
  }
  DS_HIP(hipMemcpy(m.sweep_in, pat.data(), in_bytes, hipMemcpyHostToDevice));
  return DSTACK_OK;
}

uint32_t first_slots_mask(int slots) { return slots >= 32 ? 0xFFFFFFFFu : ((1u << slots) - 1); }

// Median and p99 latency (us) of `reps` event-timed forwards after `warmup`
// on a fresh partition of the first `slots` slots.
dstack_status measure_latency(Model& m, int batch, int slots, int warmup, int reps, double* med, double* p99) {
  dstack_status s = ensure_sweep_buffers(m);
  if (s != DSTACK_OK) return s;
  dstack_partition p;
  s = make_partition(first_slots_mask(slots), &p);
  if (s != DSTACK_OK) return s;
  std::vector<float> ms(reps);
  std::vector<hipEvent_t> ev(2 * reps);
  for (auto& e : ev) {
    if (hipEventCreate(&e) != hipSuccess) e = nullptr;
  }
  for (int w = 0; w < warmup && s == DSTACK_OK; ++w)
    s = infer_impl(m, batch, m.sweep_in, m.sweep_out, p, nullptr, SWEEP_WS_ID);
  for (int r = 0; r < reps && s == DSTACK_OK; ++r) {
    (void)hipEventRecord(ev[2 * r], p->stream);
    s = infer_impl(m, batch, m.sweep_in, m.sweep_out, p, nullptr, SWEEP_WS_ID);
    (void)hipEventRecord(ev[2 * r + 1], p->stream);
  }
  hipError_t e = hipStreamSynchronize(p->stream);
  for (int r = 0; r < reps && e == hipSuccess; ++r) e = hipEventElapsedTime(&ms[r], ev[2 * r], ev[2 * r + 1]);
  for (auto& x : ev)
    if (x) (void)hipEventDestroy(x);
  dstack_partition_destroy(p);
  if (s != DSTACK_OK) return s;
  if (e != hipSuccess) return hip_fail(e, "latency timing");
  std::vector<double> us(reps);
  for (int r = 0; r < reps; ++r) us[r] = 1000.0 * ms[r];
  std::sort(us.begin(), us.end());
  *med = (reps % 2) ? us[reps / 2] : 0.5 * (us[reps / 2 - 1] + us[reps / 2]);
  *p99 = us[std::min(reps - 1, (int)std::ceil(0.99 * reps) - 1)];
  return DSTACK_OK;
}

int64_t round_us(double us) { return std::max<int64_t>(1, (int64_t)std::floor(us + 0.5)); }

}  // namespace

dstack_status dstack_kernel_shapes(dstack_model h, int batch, const void* d_in, void* d_out, dstack_partition p,
                                   dstack_kernel_shape* out, int max_units, int* n_units) {
  return guarded([&] {
    DS_CHECK(h && p && out && n_units, DSTACK_E_INVALID, "kernel_shapes: null pointer");
    DS_CHECK(max_units >= 0, DSTACK_E_INVALID, "kernel_shapes: max_units must be >= 0");
    dstack_status s = check_batch(h->m, batch);
    if (s != DSTACK_OK) return s;
    std::vector<LaunchShape> rec;
    struct Install {  // the recorder is removed on every exit path
      explicit Install(std::vector<LaunchShape>* r) { shape_recorder() = r; }
      ~Install() { shape_recorder() = nullptr; }
    } install(&rec);
    KernelTimer timer;
    timer.st = p->stream;
    timer.dry = true;
    s = infer_impl(h->m, batch, d_in, d_out, p, &timer);
    if (s != DSTACK_OK) return s;
    int n = 0;
    for (const auto& u : timer.units) {
      if (n >= max_units) break;
      dstack_kernel_shape k{};
      k.kind = u.kind;
      k.launches = (int)(u.l1 - u.l0);
      for (size_t i = u.l0; i < u.l1; ++i)
        if (rec[i].workgroups > k.workgroups) {
          k.workgroups = rec[i].workgroups;
          k.blocks_per_cu = rec[i].per_cu;
        }
      k.flops = u.flops;
      k.bytes = u.bytes;
      out[n++] = k;
    }
    *n_units = n;
    return DSTACK_OK;
  });
}

dstack_status dstack_knee_model_eval(const dstack_knee_model* m, const int* s_values, int n_s, double* et_out,
                                     int* knee_index) {
  return guarded([&] { return knee_model_eval(m, s_values, n_s, et_out, knee_index); });
}

dstack_status dstack_knee_model_sequence(int p, int b, int kmax, double* n_out) {
  return guarded([&] { return knee_model_sequence(p, b, kmax, n_out); });
}

dstack_status dstack_knee_sweep(dstack_model h, int batch, const double* fractions, int n, int warmup, int reps,
                                dstack_knee_result* out) {
  return guarded([&] {
    DS_CHECK(h && fractions && out, DSTACK_E_INVALID, "knee_sweep: null pointer");
    DS_CHECK(n >= 1 && n <= DSTACK_MAX_SWEEP && warmup >= 0 && reps >= 1, DSTACK_E_INVALID,
             "knee_sweep: n in 1..32, warmup >= 0, reps >= 1");
    Model& m = h->m;
    dstack_status s = check_batch(m, batch);
    if (s != DSTACK_OK) return s;
    std::memset(out, 0, sizeof(*out));
    out->n = n;
    out->batch = batch;
    for (int i = 0; i < n; ++i) {
      int slots;
      s = slots_from_fraction(fractions[i], &slots);
      if (s != DSTACK_OK) return s;
      double med, p99;
      s = measure_latency(m, batch, slots, warmup, reps, &med, &p99);
      if (s != DSTACK_OK) return s;
      out->slots[i] = slots;
      out->n_cu[i] = slots * DSTACK_CUS_PER_SLOT;
      out->latency_us_exact[i] = med;
      out->latency_us[i] = round_us(med);
      out->p99_us[i] = p99;
    }
    int k = knee_index(batch, out->latency_us, out->slots, n);
    out->knee_index = k;
    out->knee_slots = out->slots[k];
    out->deployed_slots = std::min(DSTACK_TOTAL_SLOTS, out->knee_slots + 2);
    return DSTACK_OK;
  });
}

namespace {

void fill_search(int batch, int total, int overprov, int knee, const std::vector<std::pair<int, int64_t>>& probes,
                 dstack_knee_search_result* out) {
  out->batch = batch;
  out->knee_slots = knee;
  out->deployed_slots = std::min(total, knee + overprov);
  out->n_probes = (int)probes.size();
  for (size_t i = 0; i < probes.size() && i < DSTACK_MAX_PROBES; ++i) {
    out->probe_slots[i] = probes[i].first;
    out->probe_latency_us[i] = probes[i].second;
  }
}

}  // namespace

dstack_status dstack_knee_search_table(int batch, const int* slots, const int64_t* latency_us, int n,
                                       int start_slots, int total, int overprov_slots,
                                       dstack_knee_search_result* out) {
  return guarded([&] {
    DS_CHECK(slots && latency_us && out, DSTACK_E_INVALID, "knee_search: null pointer");
    DS_CHECK(batch >= 1 && n >= 1 && n <= DSTACK_MAX_SWEEP && total >= 1 && total <= 64 && overprov_slots >= 0,
             DSTACK_E_INVALID, "knee_search: bad arguments");
    std::vector<int> cand(slots, slots + n);
    for (int i = 0; i < n; ++i) {
      DS_CHECK(latency_us[i] > 0 && cand[i] >= 1 && cand[i] <= total && (i == 0 || cand[i] > cand[i - 1]),
               DSTACK_E_INVALID, "knee_search: ascending slot counts in 1..total, latencies > 0");
    }
    std::memset(out, 0, sizeof(*out));
    std::vector<std::pair<int, int64_t>> probes;
    const int k = knee_search(batch, cand, start_slots, [&](int s) {
      return latency_us[std::lower_bound(cand.begin(), cand.end(), s) - cand.begin()];
    }, &probes);
    fill_search(batch, total, overprov_slots, cand[k], probes, out);
    return DSTACK_OK;
  });
}

dstack_status dstack_knee_search(dstack_model h, int batch, const double* fractions, int n, int start_slots, int warmup,
                                 int reps, dstack_knee_search_result* out) {
  return guarded([&] {
    DS_CHECK(h && fractions && out, DSTACK_E_INVALID, "knee_search: null pointer");
    DS_CHECK(n >= 1 && n <= DSTACK_MAX_SWEEP && warmup >= 0 && reps >= 1, DSTACK_E_INVALID,
             "knee_search: n in 1..32, warmup >= 0, reps >= 1");
    Model& m = h->m;
    dstack_status s = check_batch(m, batch);
    if (s != DSTACK_OK) return s;
    std::vector<int> cand;
    for (int i = 0; i < n; ++i) {
      int slots;
      s = slots_from_fraction(fractions[i], &slots);
      if (s != DSTACK_OK) return s;
      DS_CHECK(cand.empty() || slots > cand.back(), DSTACK_E_INVALID, "knee_search: fractions must ascend");
      cand.push_back(slots);
    }
    std::memset(out, 0, sizeof(*out));
    std::vector<std::pair<int, int64_t>> probes;
    dstack_status err = DSTACK_OK;
    const auto t0 = std::chrono::steady_clock::now();
    const int k = knee_search(batch, cand, start_slots, [&](int slots) -> int64_t {
      if (err != DSTACK_OK) return 1;
      double med, p99;
      err = measure_latency(m, batch, slots, warmup, reps, &med, &p99);
      return err == DSTACK_OK ? round_us(med) : 1;
    }, &probes);
    if (err != DSTACK_OK) return err;
    out->seconds = std::chrono::duration<double>(std::chrono::steady_clock::now() - t0).count();
    fill_search(batch, DSTACK_TOTAL_SLOTS, 2, cand[k], probes, out);
    return DSTACK_OK;
  });
}

dstack_status dstack_switch_probe(dstack_model h, int batch, int from_slots, int to_slots, int reps,
                                  dstack_switch_result* out) {
  return guarded([&] {
    DS_CHECK(h && out, DSTACK_E_INVALID, "switch_probe: null pointer");
    DS_CHECK(from_slots >= 1 && from_slots <= DSTACK_TOTAL_SLOTS && to_slots >= 1 && to_slots <= DSTACK_TOTAL_SLOTS &&
                 reps >= 1 && reps <= 1000,
             DSTACK_E_INVALID, "switch_probe: slots in 1..32, reps in 1..1000");
    Model& m = h->m;
    dstack_status s = check_batch(m, batch);
    if (s != DSTACK_OK) return s;
    s = ensure_sweep_buffers(m);
    if (s != DSTACK_OK) return s;
    std::memset(out, 0, sizeof(*out));
    using clk = std::chrono::steady_clock;
    auto us_since = [](clk::time_point t) { return std::chrono::duration<double, std::micro>(clk::now() - t).count(); };
    // the active partition, warmed up; its own workspace id keeps the two apart
    constexpr int ACTIVE_WS = 1, STANDBY_WS = 2;
    dstack_partition a = nullptr, b = nullptr;
    hipEvent_t e0 = nullptr, e1 = nullptr;
    auto cleanup = [&] {
      if (e0) (void)hipEventDestroy(e0);
      if (e1) (void)hipEventDestroy(e1);
      if (a) dstack_partition_destroy(a);
      if (b) dstack_partition_destroy(b);
    };
    auto run = [&](dstack_partition p, int ws) { return infer_impl(m, batch, m.sweep_in, m.sweep_out, p, nullptr, ws); };
    s = make_partition(first_slots_mask(from_slots), &a);
    for (int r = 0; r < 3 && s == DSTACK_OK; ++r) s = run(a, ACTIVE_WS);
    if (s == DSTACK_OK && hipStreamSynchronize(a->stream) != hipSuccess) s = fail(DSTACK_E_HIP, "switch_probe: sync");
    if (s != DSTACK_OK) {
      cleanup();
      return s;
    }
    // cold change: a new partition is created and its first forward captured and run
    auto t0 = clk::now();
    s = make_partition(first_slots_mask(to_slots), &b);
    out->create_us = us_since(t0);
    if (s == DSTACK_OK) s = run(b, STANDBY_WS);
    if (s == DSTACK_OK && hipStreamSynchronize(b->stream) != hipSuccess) s = fail(DSTACK_E_HIP, "switch_probe: sync");
    out->cold_us = us_since(t0);
    // active-standby: the standby is ready; after the active's batch ends the
    // host hands the next batch to the standby; gap = standby start - active end (device clock)
    if (s == DSTACK_OK && (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess))
      s = fail(DSTACK_E_HIP, "switch_probe: events");
    std::vector<double> gaps;
    for (int r = 0; r < reps && s == DSTACK_OK; ++r) {
      s = run(a, ACTIVE_WS);
      if (s != DSTACK_OK) break;
      (void)hipEventRecord(e0, a->stream);
      if (hipEventSynchronize(e0) != hipSuccess) {
        s = fail(DSTACK_E_HIP, "switch_probe: wait");
        break;
      }
      (void)hipEventRecord(e1, b->stream);
      s = run(b, STANDBY_WS);
      if (s != DSTACK_OK) break;
      if (hipStreamSynchronize(b->stream) != hipSuccess) {
        s = fail(DSTACK_E_HIP, "switch_probe: sync");
        break;
      }
      float ms = 0.f;
      (void)hipEventElapsedTime(&ms, e0, e1);
      gaps.push_back(1000.0 * ms);
    }
    if (s == DSTACK_OK) {
      double med, p99;
      s = measure_latency(m, batch, from_slots, 2, 5, &med, &p99);
      out->from_latency_us = med;
      if (s == DSTACK_OK) s = measure_latency(m, batch, to_slots, 2, 5, &med, &p99);
      out->to_latency_us = med;
    }
    cleanup();
    if (s != DSTACK_OK) return s;
    std::sort(gaps.begin(), gaps.end());
    out->standby_gap_us = gaps[gaps.size() / 2];
    out->standby_gap_max_us = gaps.back();
    return DSTACK_OK;
  });
}

dstack_status dstack_schedule(const dstack_sched_model* models, int n, const dstack_sched_params* prm,
                              dstack_schedule_out* out) {
  return guarded([&] { return schedule(models, n, prm, out); });
}

dstack_status dstack_simulate(const dstack_sched_model* models, int n, const dstack_sched_params* prm,
                              const dstack_sim_params* sim, dstack_run_out* out) {
  return guarded([&] { return simulate(models, n, prm, sim, out); });
}

dstack_status dstack_simulate_ideal(const dstack_ideal_model* models, int n, int64_t horizon_us, int64_t slot_us,
                                    int total_slots, dstack_ideal_out* out) {
  return guarded([&] { return simulate_ideal(models, n, horizon_us, slot_us, total_slots, out); });
}

dstack_status dstack_serve(const dstack_model* models, int n, const void* const* d_in, void* const* d_out,
                           const dstack_sched_model* tables, const dstack_sched_params* prm,
                           const dstack_sim_params* sim, dstack_run_out* out, dstack_job_record* log,
                           int log_capacity, int* n_log, dstack_serve_event* events, int event_capacity,
                           int* n_events) {
  return guarded([&] {
    return serve(models, n, d_in, d_out, tables, prm, sim, out, log, log_capacity, n_log, events, event_capacity,
                 n_events);
  });
}

// ----------------------------------------------------- kernel-level ops ----

// compute units a stream may run on (its CU mask; the whole device for the
// null stream or when the mask cannot be read)
static int stream_cu_count(hipStream_t st) {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess || hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    n = 256;
  if (st == nullptr) return n;
  uint32_t words[8] = {0, 0, 0, 0, 0, 0, 0, 0};
  if (hipExtStreamGetCUMask(st, 8, words) != hipSuccess) return n;
  int bits = 0;
  for (uint32_t w : words) bits += __builtin_popcount(w);
  return bits > 0 ? std::min(bits, n) : n;
}

dstack_status dstack_op_conv2d(const void* x, int N, int H, int W, int C, const void* w, int K, int R, int S,
                               int stride, int pad, const float* scale, const float* shift, const void* res, int act,
                               void* y, int out_fp32, void* stream) {
  return guarded([&] {
    DS_CHECK(x && w && y, DSTACK_E_INVALID, "conv2d: null pointer");
    DS_CHECK(act >= 0 && act <= 4, DSTACK_E_INVALID, "conv2d: act must be 0..4");
    return launch_conv2d(static_cast<const bf16*>(x), N, H, W, C, static_cast<const bf16*>(w), K, R, S, stride, pad,
                         scale, shift, static_cast<const bf16*>(res), act, y, out_fp32 != 0,
                         stream_cu_count((hipStream_t)stream), (hipStream_t)stream);
  });
}

namespace {

constexpr size_t kConvCounterBytes = SPLITK_TILE_COUNTERS * sizeof(unsigned);  // 16 KiB, 256-aligned

void fill_conv_plan(const ConvLaunchPlan& p, dstack_conv_plan* out) {
  std::memset(out, 0, sizeof(*out));
  out->kernel = p.kernel;
  out->mode = p.mode;
  out->tile_n = p.bn;
  out->tile_m = p.bm;
  out->splits = p.splits;
  out->tiles_per_split = p.kt_per_split;
  out->stages = p.stages;
  out->workspace_bytes = p.splits > 1 ? kConvCounterBytes + p.split_bytes : 0;
}

// slice bytes a workspace of `bytes` leaves after its counters
size_t slice_room(const void* ws, size_t bytes) { return ws && bytes > kConvCounterBytes ? bytes - kConvCounterBytes : 0; }

}  // namespace

dstack_status dstack_conv2d_plan(int N, int H, int W, int C, int K, int R, int S, int stride, int pad, int act,
                                 int out_fp32, int n_cu, size_t workspace_bytes, dstack_conv_plan* out) {
  return guarded([&] {
    DS_CHECK(out, DSTACK_E_INVALID, "conv2d_plan: null pointer");
    ConvLaunchPlan p;
    dstack_status s = conv2d_plan(N, H, W, C, K, R, S, stride, pad, act, out_fp32 != 0, n_cu,
                                  workspace_bytes > kConvCounterBytes ? workspace_bytes - kConvCounterBytes : 0, &p);
    if (s != DSTACK_OK) return s;
    fill_conv_plan(p, out);
    return DSTACK_OK;
  });
}

dstack_status dstack_op_conv2d_ws(const void* x, int N, int H, int W, int C, const void* w, int K, int R, int S,
                                  int stride, int pad, const float* scale, const float* shift, const void* res,
                                  int act, void* y, int out_fp32, int n_cu, void* workspace, size_t workspace_bytes,
                                  void* stream) {
  return guarded([&] {
    DS_CHECK(x && w && y, DSTACK_E_INVALID, "conv2d_ws: null pointer");
    DS_CHECK(act >= 0 && act <= 4, DSTACK_E_INVALID, "conv2d_ws: act must be 0..4");
    DS_CHECK(!workspace || ((uintptr_t)workspace % 256) == 0, DSTACK_E_INVALID,
             "conv2d_ws: workspace must be 256-byte aligned");
    const int cus = n_cu > 0 ? n_cu : stream_cu_count((hipStream_t)stream);
    char* base = static_cast<char*>(workspace);
    const size_t room = slice_room(workspace, workspace_bytes);
    return launch_conv2d_ws(static_cast<const bf16*>(x), N, H, W, C, static_cast<const bf16*>(w), K, R, S, stride,
                            pad, scale, shift, static_cast<const bf16*>(res), act, y, out_fp32 != 0, cus,
                            room ? reinterpret_cast<float*>(base + kConvCounterBytes) : nullptr, room,
                            room ? reinterpret_cast<unsigned*>(base) : nullptr, (hipStream_t)stream);
  });
}

dstack_status dstack_op_conv2d_noalloc(const void* x, int N, int H, int W, int C, const void* w, int K, int R, int S,
                                       int stride, int pad, const float* scale, const float* shift, const void* res,
                                       int act, void* y, int out_fp32, int n_cu, void* stream) {
  return guarded([&] {
    DS_CHECK(x && w && y, DSTACK_E_INVALID, "conv2d_noalloc: null pointer");
    DS_CHECK(act >= 0 && act <= 4, DSTACK_E_INVALID, "conv2d_noalloc: act must be 0..4");
    const int cus = n_cu > 0 ? n_cu : stream_cu_count((hipStream_t)stream);
    return launch_conv2d_noalloc(static_cast<const bf16*>(x), N, H, W, C, static_cast<const bf16*>(w), K, R, S,
                                 stride, pad, scale, shift, static_cast<const bf16*>(res), act, y, out_fp32 != 0, cus,
                                 (hipStream_t)stream);
  });
}

size_t dstack_conv2d_noalloc_scratch_bytes(void) { return CONV_SCRATCH_BYTES; }

dstack_status dstack_arch_convs(const char* arch, int batch, dstack_conv_shape* out, int max_convs, int* n_convs) {
  return guarded([&] {
    DS_CHECK(arch && n_convs && (out || max_convs == 0), DSTACK_E_INVALID, "arch_convs: null pointer");
    Model m;
    dstack_status s = build_arch(arch, m);
    if (s != DSTACK_OK) return s;
    DS_CHECK(batch >= 1 && batch <= m.max_batch, DSTACK_E_INVALID, "arch_convs: batch out of range");
    int n = 0;
    auto put = [&](const dstack_conv_shape& c) {
      if (n < max_convs) out[n] = c;
      ++n;
    };
    for (const Op& op : m.ops) {
      if (op.kind == OP_CONV) {
        put(dstack_conv_shape{batch, op.H, op.W, op.C, op.K, op.R, op.S, op.stride, op.pad, op.act,
                              op.res != BUF_NONE ? 1 : 0, 0});
      } else if (op.kind == OP_LSTM) {  // the input projection of all steps: a 1x1 convolution with fp32 output
        put(dstack_conv_shape{op.T * batch, 1, 1, op.I, 4 * op.Hd, 1, 1, 1, 0, ACT_NONE, 0, 1});
      }
    }
    *n_convs = n;
    return DSTACK_OK;
  });
}

dstack_status dstack_op_conv2d_rgb(const void* x, int N, int H, int W, const void* w4, int K, int R, int stride,
                                   int pad, const float* scale, const float* shift, int act, void* y, void* stream) {
  return guarded([&] {
    DS_CHECK(x && w4 && y, DSTACK_E_INVALID, "conv2d_rgb: null pointer");
    DS_CHECK(act >= 0 && act <= 2, DSTACK_E_INVALID, "conv2d_rgb: act must be 0, 1 or 2");
    return launch_conv2d_rgb(static_cast<const bf16*>(x), N, H, W, static_cast<const bf16*>(w4), K, R, stride, pad,
                             scale, shift, act, static_cast<bf16*>(y), (hipStream_t)stream);
  });
}

dstack_status dstack_op_expand_dw(const void* x, int N, int H, int W, int Cin, const void* we, int Ce,
                                  const float* se, const float* he, int act_e, const void* wd, int stride,
                                  const float* sd, const float* hd, int act_d, void* y, void* stream) {
  return guarded([&] {
    return launch_expand_dw(static_cast<const bf16*>(x), N, H, W, Cin, static_cast<const bf16*>(we), Ce, se, he,
                            act_e, static_cast<const bf16*>(wd), stride, sd, hd, act_d, static_cast<bf16*>(y),
                            (hipStream_t)stream);
  });
}

dstack_status dstack_op_dwconv3x3(const void* x, int N, int H, int W, int C, const void* w, int stride,
                                  const float* scale, const float* shift, int act, void* y, void* stream) {
  return guarded([&] {
    DS_CHECK(x && w && y && scale && shift, DSTACK_E_INVALID, "dwconv3x3: null pointer");
    DS_CHECK(act >= 0 && act <= 2, DSTACK_E_INVALID, "dwconv3x3: act must be 0, 1 or 2");
    return launch_dwconv3x3(static_cast<const bf16*>(x), N, H, W, C, static_cast<const bf16*>(w), stride, scale,
                            shift, act, static_cast<bf16*>(y), (hipStream_t)stream);
  });
}

size_t dstack_fc_workspace_bytes(int B, int I, int O) {
  if (B < 1 || I < 1 || O < 1) return 0;
  return fc_workspace_bytes(B, I, O, 256);
}

dstack_status dstack_op_fc(const void* x, int B, int I, const void* w, const float* bias, int O, int act, void* y,
                           int out_fp32, void* workspace, size_t workspace_bytes, void* stream) {
  return guarded([&] {
    DS_CHECK(x && w && y, DSTACK_E_INVALID, "fc: null pointer");
    DS_CHECK(act >= 0 && act <= 2, DSTACK_E_INVALID, "fc: act must be 0, 1 or 2");
    return launch_fc(static_cast<const bf16*>(x), B, I, static_cast<const bf16*>(w), bias, O, act, y, out_fp32 != 0,
                     256, static_cast<float*>(workspace), workspace ? workspace_bytes : 0, (hipStream_t)stream);
  });
}

dstack_status dstack_op_maxpool(const void* x, int N, int H, int W, int C, int k, int stride, int pad, void* y,
                                void* stream) {
  return guarded([&] {
    DS_CHECK(x && y, DSTACK_E_INVALID, "maxpool: null pointer");
    return launch_maxpool(static_cast<const bf16*>(x), N, H, W, C, k, stride, pad, static_cast<bf16*>(y),
                          (hipStream_t)stream);
  });
}

dstack_status dstack_op_avgpool(const void* x, int N, int H, int W, int C, void* y, void* stream) {
  return guarded([&] {
    DS_CHECK(x && y, DSTACK_E_INVALID, "avgpool: null pointer");
    return launch_avgpool(static_cast<const bf16*>(x), N, H, W, C, static_cast<bf16*>(y), (hipStream_t)stream);
  });
}

// gx [T][B][4H] fp32 | c [B][H] fp32 | W_hh in fragment order [4H][H] bf16 |
// h(t-1), h(t) in fragment order [2][B][H] bf16, each part 256-byte aligned
static size_t align256z(size_t n) { return (n + 255) / 256 * 256; }
size_t dstack_lstm_workspace_bytes(int T, int B, int H) {
  if (T <= 0 || B <= 0 || H <= 0) return 0;
  return align256z((size_t)T * B * 4 * H * 4) + align256z((size_t)B * H * 4) + align256z((size_t)4 * H * H * 2) +
         (size_t)2 * B * H * 2;
}

dstack_status dstack_op_lstm_layer(const void* x, int T, int B, int I, int H, const void* w_ih, const void* w_hh,
                                   const float* bias, void* h_bf16, float* h_f32, void* workspace, void* stream) {
  return guarded([&] {
    DS_CHECK(x && w_ih && w_hh && bias && h_bf16 && workspace, DSTACK_E_INVALID, "lstm_layer: null pointer");
    DS_CHECK(T >= 1 && I % 8 == 0 && I > 0, DSTACK_E_UNSUPPORTED, "lstm_layer: T >= 1, I % 8 == 0");
    DS_CHECK(B >= 1 && B <= 32, DSTACK_E_UNSUPPORTED, "lstm_layer: batch must be 1..32");
    DS_CHECK(H >= 32 && H % 32 == 0 && H <= 2048, DSTACK_E_UNSUPPORTED, "lstm_layer: H must be a multiple of 32, <= 2048");
    char* p = static_cast<char*>(workspace);
    float* gx = reinterpret_cast<float*>(p);
    p += align256z((size_t)T * B * 4 * H * 4);
    float* c = reinterpret_cast<float*>(p);
    p += align256z((size_t)B * H * 4);
    bf16* wp = reinterpret_cast<bf16*>(p);
    p += align256z((size_t)4 * H * H * 2);
    bf16* hp = reinterpret_cast<bf16*>(p);
    return lstm_layer_run(static_cast<const bf16*>(x), T, B, I, H, static_cast<const bf16*>(w_ih),
                          static_cast<const bf16*>(w_hh), nullptr, bias, static_cast<bf16*>(h_bf16), h_f32, gx, c,
                          wp, hp, stream_cu_count((hipStream_t)stream), (hipStream_t)stream, nullptr);
  });
}

dstack_status dstack_op_embed_ln(const int32_t* ids, int rows, int T, int vocab, const void* we, const void* pe,
                                 const void* te, int H, const float* gamma, const float* beta, float eps, void* y,
                                 void* stream) {
  return guarded([&] {
    return launch_embed_ln(ids, rows, T, vocab, static_cast<const bf16*>(we), static_cast<const bf16*>(pe),
                           static_cast<const bf16*>(te), H, gamma, beta, eps, static_cast<bf16*>(y),
                           (hipStream_t)stream);
  });
}

dstack_status dstack_op_layernorm(const void* x, int rows, int H, const float* gamma, const float* beta, float eps,
                                  void* y, void* stream) {
  return guarded([&] {
    return launch_layernorm(static_cast<const bf16*>(x), rows, H, gamma, beta, eps, static_cast<bf16*>(y),
                            (hipStream_t)stream);
  });
}

dstack_status dstack_op_attention(const void* qkv, int B, int T, int heads, int dh, void* out, void* stream) {
  return guarded([&] {
    return launch_attention(static_cast<const bf16*>(qkv), B, T, heads, dh, static_cast<bf16*>(out),
                            (hipStream_t)stream);
  });
}

}  // extern "C"

// Launcher-internal entry points (C++ linkage; see launcher.hpp).
namespace dstack {

dstack_status launcher_infer(dstack_model h, int batch, const void* d_in, void* d_out, dstack_partition p,
                             int ws_id) {
  return guarded([&] {
    DS_CHECK(h && ws_id >= kLauncherWsBase && ws_id < kLauncherWsBase + kLauncherWsCount, DSTACK_E_INVALID,
             "launcher: bad model or workspace id");
    return infer_impl(h->m, batch, d_in, d_out, p, nullptr, ws_id);
  });
}

dstack_status launcher_prepare(dstack_model h, int batch, const void* d_in, void* d_out, dstack_partition p, int n_cu,
                               int ws_id) {
  return guarded([&] {
    DS_CHECK(h && ws_id >= kLauncherWsBase && ws_id < kLauncherWsBase + kLauncherWsCount && n_cu >= 1,
             DSTACK_E_INVALID, "launcher: bad model, workspace id or CU count");
    return infer_impl(h->m, batch, d_in, d_out, p, nullptr, ws_id, n_cu);
  });
}

}  // namespace dstack
