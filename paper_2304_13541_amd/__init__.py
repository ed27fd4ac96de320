"""Python binding of libdstack (argument marshalling only).

Every computation runs in the HIP library behind the C ABI declared in
``include/dstack.h``; this module only converts arguments, checks status
codes and wraps PyTorch device tensors and streams.  It raises if the
compiled library is missing: there is no fallback path.
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# DSTACK_LIBRARY may name another build of the same sources (the CPU
# sanitizer build libdstack_san.so); the default is the in-tree library.
LIB_PATH = os.environ.get("DSTACK_LIBRARY") or os.path.join(HERE, "libdstack.so")

OK, E_INVALID, E_UNSUPPORTED, E_HIP, E_OOM, E_INFEASIBLE, E_STATE = 0, -1, -2, -3, -4, -5, -6
TOTAL_SLOTS = 32
CUS_PER_SLOT = 8
MAX_SWEEP, MAX_BATCHES, MAX_MODELS, MAX_JOBS = 32, 8, 16, 512
ARCHS = ("tinycnn", "resnet50", "mobilenetv2", "vgg19", "lstm2", "bert", "bert_long")
KIND_NAMES = {0: "mfma", 1: "depthwise", 2: "fc", 3: "lstm_step", 4: "glue", 5: "direct_conv", 6: "expand_dw",
              7: "attention"}


class DStackError(RuntimeError):
    def __init__(self, status, msg):
        super().__init__("dstack status %d: %s" % (status, msg))
        self.status = status


class ModelInfo(ctypes.Structure):
    _fields_ = [("arch", ctypes.c_char * 16), ("is_lstm", ctypes.c_int), ("max_batch", ctypes.c_int),
                ("in_h", ctypes.c_int), ("in_w", ctypes.c_int), ("in_c", ctypes.c_int),
                ("seq_len", ctypes.c_int), ("in_features", ctypes.c_int), ("out_features", ctypes.c_int),
                ("num_tensors", ctypes.c_int), ("num_params", ctypes.c_int64), ("num_kernels", ctypes.c_int),
                ("flops_per_item", ctypes.c_double), ("mfma_flops_per_item", ctypes.c_double),
                ("weight_bytes", ctypes.c_double), ("input_tokens", ctypes.c_int)]


class LayerTime(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int), ("ms", ctypes.c_float), ("flops", ctypes.c_double), ("bytes", ctypes.c_double),
                ("gemm_m", ctypes.c_int), ("gemm_n", ctypes.c_int), ("gemm_k", ctypes.c_int)]


class KernelShape(ctypes.Structure):
    _fields_ = [("kind", ctypes.c_int), ("launches", ctypes.c_int), ("workgroups", ctypes.c_int64),
                ("blocks_per_cu", ctypes.c_int), ("pad", ctypes.c_int), ("flops", ctypes.c_double),
                ("bytes", ctypes.c_double)]


class KneeModel(ctypes.Structure):
    _fields_ = [("n_kernels", ctypes.c_int), ("pad", ctypes.c_int), ("n_par", ctypes.POINTER(ctypes.c_double)),
                ("t_p", ctypes.POINTER(ctypes.c_double)), ("reps", ctypes.POINTER(ctypes.c_double)),
                ("data", ctypes.POINTER(ctypes.c_double)), ("t_np", ctypes.c_double),
                ("mem_bw_per_sm", ctypes.c_double), ("batch_serial", ctypes.c_double)]


class KneeResult(ctypes.Structure):
    _fields_ = [("n", ctypes.c_int), ("batch", ctypes.c_int), ("slots", ctypes.c_int * MAX_SWEEP),
                ("n_cu", ctypes.c_int * MAX_SWEEP), ("latency_us", ctypes.c_int64 * MAX_SWEEP),
                ("latency_us_exact", ctypes.c_double * MAX_SWEEP), ("p99_us", ctypes.c_double * MAX_SWEEP),
                ("knee_index", ctypes.c_int), ("knee_slots", ctypes.c_int), ("deployed_slots", ctypes.c_int)]


MAX_PROBES = 64


class KneeSearchResult(ctypes.Structure):
    _fields_ = [("batch", ctypes.c_int), ("knee_slots", ctypes.c_int), ("deployed_slots", ctypes.c_int),
                ("n_probes", ctypes.c_int), ("probe_slots", ctypes.c_int * MAX_PROBES),
                ("probe_latency_us", ctypes.c_int64 * MAX_PROBES), ("seconds", ctypes.c_double)]


class SwitchResult(ctypes.Structure):
    _fields_ = [(n, ctypes.c_double) for n in ("create_us", "cold_us", "standby_gap_us", "standby_gap_max_us",
                                               "from_latency_us", "to_latency_us")]


class SchedModel(ctypes.Structure):
    _fields_ = [("slo_us", ctypes.c_int64), ("max_batch", ctypes.c_int), ("rate_per_s", ctypes.c_int),
                ("n_batches", ctypes.c_int), ("batches", ctypes.c_int * MAX_BATCHES), ("n_slots", ctypes.c_int),
                ("slots", ctypes.c_int * MAX_SWEEP), ("latency_us", (ctypes.c_int64 * MAX_SWEEP) * MAX_BATCHES)]


class SchedParams(ctypes.Structure):
    _fields_ = [("period_us", ctypes.c_int64), ("total_slots", ctypes.c_int), ("overprov_slots", ctypes.c_int),
                ("placement", ctypes.c_int)]


class Job(ctypes.Structure):
    _fields_ = [("model", ctypes.c_int), ("k", ctypes.c_int), ("release_us", ctypes.c_int64),
                ("deadline_us", ctypes.c_int64), ("start_us", ctypes.c_int64), ("duration_us", ctypes.c_int64),
                ("slots", ctypes.c_int), ("missed", ctypes.c_int), ("slot_mask", ctypes.c_uint64)]


class ScheduleOut(ctypes.Structure):
    _fields_ = [("n_models", ctypes.c_int), ("batch", ctypes.c_int * MAX_MODELS),
                ("knee_slots", ctypes.c_int * MAX_MODELS), ("deployed_slots", ctypes.c_int * MAX_MODELS),
                ("latency_us", ctypes.c_int64 * MAX_MODELS), ("feasible", ctypes.c_int * MAX_MODELS),
                ("n_jobs", ctypes.c_int), ("jobs", Job * MAX_JOBS), ("utilisation_ppm", ctypes.c_int64),
                ("home_offset", ctypes.c_int * MAX_MODELS)]


class SimParams(ctypes.Structure):
    _fields_ = [("duration_us", ctypes.c_int64), ("fod", ctypes.c_int), ("sessions_window", ctypes.c_int),
                ("arrivals_us", ctypes.POINTER(ctypes.c_int64) * MAX_MODELS), ("n_arrivals", ctypes.c_int * MAX_MODELS),
                ("policy", ctypes.c_int), ("resize_violations", ctypes.c_int), ("slice_cycle_us", ctypes.c_int64)]


class ServeEvent(ctypes.Structure):
    _fields_ = [("t_us", ctypes.c_int64), ("value_us", ctypes.c_int64), ("slot_mask", ctypes.c_uint64),
                ("kind", ctypes.c_int), ("model", ctypes.c_int)]


class IdealModel(ctypes.Structure):
    _fields_ = [("n_kernels", ctypes.c_int), ("batch", ctypes.c_int), ("slots", ctypes.POINTER(ctypes.c_int)),
                ("dur_us", ctypes.POINTER(ctypes.c_int64)), ("slo_us", ctypes.c_int64)]


class IdealOut(ctypes.Structure):
    _fields_ = [("n_models", ctypes.c_int)] + [(n, ctypes.c_int64 * MAX_MODELS) for n in
                                               ("items", "forwards", "late", "busy_slot_us")] + \
               [("utilisation_ppm", ctypes.c_int64), ("hash", ctypes.c_uint64)]


class ModelStats(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int64) for n in ("served", "violations", "unserved", "planned_runs", "fod_runs",
                                               "busy_us", "p50_us", "p99_us", "plan_skips", "resizes",
                                               "final_slots")]


class JobRecord(ctypes.Structure):
    _fields_ = [("start_us", ctypes.c_int64), ("end_us", ctypes.c_int64), ("gpu_us", ctypes.c_int64),
                ("table_us", ctypes.c_int64), ("model", ctypes.c_int), ("batch", ctypes.c_int),
                ("kind", ctypes.c_int), ("slot_mask", ctypes.c_uint64)]


class RunOut(ctypes.Structure):
    _fields_ = [("n_models", ctypes.c_int), ("models", ModelStats * MAX_MODELS), ("utilisation_ppm", ctypes.c_int64),
                ("job_hash", ctypes.c_uint64), ("last_end_us", ctypes.c_int64)]


class ConvPlan(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in ("kernel", "mode", "tile_n", "tile_m", "splits", "tiles_per_split",
                                            "stages", "pad")] + [("workspace_bytes", ctypes.c_size_t)]


class ConvShape(ctypes.Structure):
    _fields_ = [(n, ctypes.c_int) for n in ("N", "H", "W", "C", "K", "R", "S", "stride", "pad", "act",
                                            "has_residual", "out_fp32")]


_lib = None
_vp, _i, _d, _u64, _sz = ctypes.c_void_p, ctypes.c_int, ctypes.c_double, ctypes.c_uint64, ctypes.c_size_t
_fp = ctypes.POINTER(ctypes.c_float)

_SIGS = {
    "dstack_last_error": ([], ctypes.c_char_p),
    "dstack_fraction_to_slots": ([_d, ctypes.POINTER(_i)], _i),
    "dstack_partition_create": ([_d, ctypes.POINTER(_vp)], _i),
    "dstack_partition_create_at": ([_i, _i, ctypes.POINTER(_vp)], _i),
    "dstack_partition_create_mask": ([ctypes.c_uint32, ctypes.POINTER(_vp)], _i),
    "dstack_partition_query": ([_vp, ctypes.POINTER(_i), ctypes.POINTER(ctypes.c_uint32), ctypes.POINTER(_vp)], _i),
    "dstack_synchronize": ([_vp], _i),
    "dstack_partition_count": ([ctypes.POINTER(_i), ctypes.POINTER(_i)], _i),
    "dstack_partition_destroy": ([_vp], None),
    "dstack_probe_cu_ids": ([_vp, _i, _i, ctypes.POINTER(ctypes.c_uint32)], _i),
    "dstack_model_load": ([ctypes.c_char_p, _u64, ctypes.POINTER(_vp)], _i),
    "dstack_model_query": ([_vp, ctypes.POINTER(ModelInfo)], _i),
    "dstack_model_export_params": ([_vp, _i, _vp, _sz], _i),
    "dstack_model_destroy": ([_vp], None),
    "dstack_generate_params": ([ctypes.c_char_p, _u64, _i, _vp, _sz, ctypes.POINTER(ctypes.c_int64)], _i),
    "dstack_infer": ([_vp, _i, _vp, _vp, _vp], _i),
    "dstack_infer_hidden": ([_vp, _i, _vp, _i, _vp, _vp], _i),
    "dstack_profile_layers": ([_vp, _i, _vp, _vp, _vp, ctypes.POINTER(LayerTime), _i, ctypes.POINTER(_i)], _i),
    "dstack_kernel_shapes": ([_vp, _i, _vp, _vp, _vp, ctypes.POINTER(KernelShape), _i, ctypes.POINTER(_i)], _i),
    "dstack_knee_model_eval": ([ctypes.POINTER(KneeModel), ctypes.POINTER(_i), _i, ctypes.POINTER(_d),
                                ctypes.POINTER(_i)], _i),
    "dstack_knee_model_sequence": ([_i, _i, _i, ctypes.POINTER(_d)], _i),
    "dstack_knee_sweep": ([_vp, _i, ctypes.POINTER(_d), _i, _i, _i, ctypes.POINTER(KneeResult)], _i),
    "dstack_schedule": ([ctypes.POINTER(SchedModel), _i, ctypes.POINTER(SchedParams), ctypes.POINTER(ScheduleOut)], _i),
    "dstack_simulate": ([ctypes.POINTER(SchedModel), _i, ctypes.POINTER(SchedParams), ctypes.POINTER(SimParams),
                         ctypes.POINTER(RunOut)], _i),
    "dstack_simulate_ideal": ([ctypes.POINTER(IdealModel), _i, ctypes.c_int64, ctypes.c_int64, _i,
                               ctypes.POINTER(IdealOut)], _i),
    "dstack_knee_search_table": ([_i, ctypes.POINTER(_i), ctypes.POINTER(ctypes.c_int64), _i, _i, _i, _i,
                                  ctypes.POINTER(KneeSearchResult)], _i),
    "dstack_knee_search": ([_vp, _i, ctypes.POINTER(_d), _i, _i, _i, _i, ctypes.POINTER(KneeSearchResult)], _i),
    "dstack_switch_probe": ([_vp, _i, _i, _i, _i, ctypes.POINTER(SwitchResult)], _i),
    "dstack_serve": ([ctypes.POINTER(_vp), _i, ctypes.POINTER(_vp), ctypes.POINTER(_vp), ctypes.POINTER(SchedModel),
                      ctypes.POINTER(SchedParams), ctypes.POINTER(SimParams), ctypes.POINTER(RunOut),
                      ctypes.POINTER(JobRecord), _i, ctypes.POINTER(_i), ctypes.POINTER(ServeEvent), _i,
                      ctypes.POINTER(_i)], _i),
    "dstack_op_conv2d": ([_vp, _i, _i, _i, _i, _vp, _i, _i, _i, _i, _i, _vp, _vp, _vp, _i, _vp, _i, _vp], _i),
    "dstack_op_conv2d_ws": ([_vp, _i, _i, _i, _i, _vp, _i, _i, _i, _i, _i, _vp, _vp, _vp, _i, _vp, _i, _i, _vp, _sz,
                             _vp], _i),
    "dstack_op_conv2d_noalloc": ([_vp, _i, _i, _i, _i, _vp, _i, _i, _i, _i, _i, _vp, _vp, _vp, _i, _vp, _i, _i, _vp],
                                 _i),
    "dstack_conv2d_noalloc_scratch_bytes": ([], _sz),
    "dstack_conv2d_plan": ([_i, _i, _i, _i, _i, _i, _i, _i, _i, _i, _i, _i, _sz, ctypes.POINTER(ConvPlan)], _i),
    "dstack_arch_convs": ([ctypes.c_char_p, _i, ctypes.POINTER(ConvShape), _i, ctypes.POINTER(_i)], _i),
    "dstack_op_conv2d_rgb": ([_vp, _i, _i, _i, _vp, _i, _i, _i, _i, _vp, _vp, _i, _vp, _vp], _i),
    "dstack_op_dwconv3x3": ([_vp, _i, _i, _i, _i, _vp, _i, _vp, _vp, _i, _vp, _vp], _i),
    "dstack_op_expand_dw": ([_vp, _i, _i, _i, _i, _vp, _i, _vp, _vp, _i, _vp, _i, _vp, _vp, _i, _vp, _vp], _i),
    "dstack_fc_workspace_bytes": ([_i, _i, _i], _sz),
    "dstack_op_fc": ([_vp, _i, _i, _vp, _vp, _i, _i, _vp, _i, _vp, _sz, _vp], _i),
    "dstack_op_maxpool": ([_vp, _i, _i, _i, _i, _i, _i, _i, _vp, _vp], _i),
    "dstack_op_avgpool": ([_vp, _i, _i, _i, _i, _vp, _vp], _i),
    "dstack_lstm_workspace_bytes": ([_i, _i, _i], _sz),
    "dstack_op_embed_ln": ([_vp, _i, _i, _i, _vp, _vp, _vp, _i, _vp, _vp, ctypes.c_float, _vp, _vp], _i),
    "dstack_op_layernorm": ([_vp, _i, _i, _vp, _vp, ctypes.c_float, _vp, _vp], _i),
    "dstack_op_attention": ([_vp, _i, _i, _i, _i, _vp, _vp], _i),
    "dstack_op_lstm_layer": ([_vp, _i, _i, _i, _i, _vp, _vp, _vp, _vp, _vp, _vp, _vp], _i),
}


def lib():
    """Load libdstack.so (built in-tree by paper_2304_13541_amd/build.py)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise ImportError("libdstack.so is not built (run __graft_entry__.build()); there is no fallback path")
        try:  # PyTorch bundles a HIP runtime with the same soname: load it first so one runtime serves both
            import torch  # noqa: F401
        except ImportError:
            pass
        L = ctypes.CDLL(LIB_PATH)
        for name, (args, res) in _SIGS.items():
            f = getattr(L, name)
            f.argtypes = args
            f.restype = res
        _lib = L
    return _lib


def _check(st):
    if st != OK:
        raise DStackError(st, lib().dstack_last_error().decode())
    return st


def _ptr(t):
    """Device pointer of a torch tensor (or None)."""
    if t is None:
        return None
    return ctypes.c_void_p(t.data_ptr())


def fraction_to_slots(f):
    s = ctypes.c_int()
    _check(lib().dstack_fraction_to_slots(float(f), ctypes.byref(s)))
    return s.value


class Partition:
    """A CU-masked HIP stream owning 8 CUs (one per XCD) per slot."""

    def __init__(self, fraction=None, slot_offset=None, n_slots=None, slot_mask=None):
        h = ctypes.c_void_p()
        if slot_mask is not None:
            _check(lib().dstack_partition_create_mask(ctypes.c_uint32(slot_mask), ctypes.byref(h)))
        elif slot_offset is not None:
            _check(lib().dstack_partition_create_at(slot_offset, n_slots, ctypes.byref(h)))
        else:
            _check(lib().dstack_partition_create(float(fraction), ctypes.byref(h)))
        self.h = h
        n = ctypes.c_int()
        words = (ctypes.c_uint32 * 8)()
        st = ctypes.c_void_p()
        _check(lib().dstack_partition_query(h, ctypes.byref(n), words, ctypes.byref(st)))
        self.n_cu = n.value
        self.mask_words = list(words)
        self.stream_ptr = st.value or 0

    def torch_stream(self, device="cuda:0"):
        import torch
        return torch.cuda.ExternalStream(self.stream_ptr, device=device)

    def synchronize(self):
        _check(lib().dstack_synchronize(self.h))

    def probe_cu_ids(self, n_blocks=4096, via_graph=False):
        out = (ctypes.c_uint32 * (2 * n_blocks))()
        _check(lib().dstack_probe_cu_ids(self.h, n_blocks, int(via_graph), out))
        return np.frombuffer(out, dtype=np.uint32).reshape(n_blocks, 2).copy()

    def destroy(self):
        if self.h:
            lib().dstack_partition_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass


class Model:
    """A random-weight model of one architecture, weights resident in HBM."""

    def __init__(self, arch, seed):
        h = ctypes.c_void_p()
        _check(lib().dstack_model_load(arch.encode(), ctypes.c_uint64(seed), ctypes.byref(h)))
        self.h = h
        self.arch = arch
        self.seed = seed
        info = ModelInfo()
        _check(lib().dstack_model_query(h, ctypes.byref(info)))
        self.info = info

    def destroy(self):
        if self.h:
            lib().dstack_model_destroy(self.h)
            self.h = None

    def __del__(self):
        try:
            self.destroy()
        except Exception:
            pass

    def input_shape(self, batch):
        """Shape of the input tensor: CNN [b,H,W,3] bf16, LSTM [T,b,I] bf16, transformer [b,T] int32 ids."""
        i = self.info
        if i.input_tokens:
            return (batch, i.seq_len)
        return (i.seq_len, batch, i.in_features) if i.is_lstm else (batch, i.in_h, i.in_w, i.in_c)

    def output_shape(self, batch):
        i = self.info
        return (i.seq_len, batch, i.out_features) if i.is_lstm else (batch, i.out_features)

    def export_params(self, idx):
        n = ctypes.c_int64()
        _check(lib().dstack_generate_params(self.arch.encode(), ctypes.c_uint64(self.seed), idx, None, 0,
                                            ctypes.byref(n)))
        out = np.empty(n.value, dtype=np.uint16)
        _check(lib().dstack_model_export_params(self.h, idx, out.ctypes.data, out.nbytes))
        return out

    def infer(self, batch, x, y, partition):
        """x: bf16 device tensor, y: fp32 device tensor; async on the partition's stream."""
        _check(lib().dstack_infer(self.h, batch, _ptr(x), _ptr(y), partition.h))

    def infer_hidden(self, batch, x, hidden, partition, layer=-1):
        """Transformer: the hidden state after encoder layer `layer` (0: embeddings; -1: the last)
        into `hidden` (bf16 [batch, T, 768])."""
        _check(lib().dstack_infer_hidden(self.h, batch, _ptr(x), int(layer), _ptr(hidden), partition.h))

    def profile_layers(self, batch, x, y, partition, max_layers=512):
        arr = (LayerTime * max_layers)()
        n = ctypes.c_int()
        _check(lib().dstack_profile_layers(self.h, batch, _ptr(x), _ptr(y), partition.h, arr, max_layers,
                                           ctypes.byref(n)))
        return [dict(kind=arr[i].kind, ms=arr[i].ms, flops=arr[i].flops, bytes=arr[i].bytes,
                     gemm=(arr[i].gemm_m, arr[i].gemm_n, arr[i].gemm_k)) for i in range(n.value)]

    def kernel_shapes(self, batch, x, y, partition, max_units=4096):
        """Per timed unit of profile_layers: kind, launches, workgroups of the largest launch,
        workgroups one CU holds at once, FLOPs and bytes; launches nothing (see dstack_kernel_shapes)."""
        arr = (KernelShape * max_units)()
        n = ctypes.c_int()
        _check(lib().dstack_kernel_shapes(self.h, batch, _ptr(x), _ptr(y), partition.h, arr, max_units,
                                          ctypes.byref(n)))
        return [dict(kind=arr[i].kind, launches=arr[i].launches, workgroups=arr[i].workgroups,
                     blocks_per_cu=arr[i].blocks_per_cu, flops=arr[i].flops, bytes=arr[i].bytes)
                for i in range(n.value)]

    def knee_search(self, batch, fractions=None, start_slots=10, warmup=5, reps=20):
        """Binary-search the knee from live latency over the GPU% grid (see dstack_knee_search)."""
        fractions = fractions or [0.1 * i for i in range(1, 11)]
        fr = (_d * len(fractions))(*fractions)
        r = KneeSearchResult()
        _check(lib().dstack_knee_search(self.h, batch, fr, len(fractions), start_slots, warmup, reps, ctypes.byref(r)))
        return _search_dict(r)

    def switch_probe(self, batch, from_slots, to_slots, reps=10):
        """Cost of a GPU% change, cold and active-standby (see dstack_switch_probe)."""
        r = SwitchResult()
        _check(lib().dstack_switch_probe(self.h, batch, from_slots, to_slots, reps, ctypes.byref(r)))
        return dict((f, getattr(r, f)) for f, _ in SwitchResult._fields_)

    def knee_sweep(self, batch, fractions, warmup=5, reps=20):
        fr = (ctypes.c_double * len(fractions))(*fractions)
        r = KneeResult()
        _check(lib().dstack_knee_sweep(self.h, batch, fr, len(fractions), warmup, reps, ctypes.byref(r)))
        n = r.n
        return dict(batch=r.batch, slots=list(r.slots[:n]), n_cu=list(r.n_cu[:n]),
                    latency_us=list(r.latency_us[:n]), latency_us_exact=list(r.latency_us_exact[:n]),
                    p99_us=list(r.p99_us[:n]), knee_index=r.knee_index, knee_slots=r.knee_slots,
                    deployed_slots=r.deployed_slots)


def _search_dict(r):
    n = min(r.n_probes, MAX_PROBES)
    return dict(batch=r.batch, knee_slots=r.knee_slots, deployed_slots=r.deployed_slots, n_probes=r.n_probes,
                probes=[(r.probe_slots[i], r.probe_latency_us[i]) for i in range(n)], seconds=r.seconds)


def knee_model_sequence(p, b, kmax):
    """N_1..N_kmax of the analytical model's synthetic kernel sequence (host only)."""
    out = (_d * kmax)()
    _check(lib().dstack_knee_model_sequence(p, b, kmax, out))
    return list(out)


def knee_model_eval(n_par, t_p, s_values, t_np, batch_serial=1.0, reps=None, data=None, mem_bw_per_sm=0.0):
    """E_t on each candidate S and the knee index of the analytical model (host only)."""
    k = len(n_par)
    arr = lambda v: None if v is None else (_d * k)(*[float(x) for x in v])
    npar, tp, rp, dt = arr(n_par), arr(t_p), arr(reps), arr(data)
    m = KneeModel(k, 0, npar, tp, rp, dt, float(t_np), float(mem_bw_per_sm), float(batch_serial))
    sv = (_i * len(s_values))(*s_values)
    et = (_d * len(s_values))()
    ki = _i()
    _check(lib().dstack_knee_model_eval(ctypes.byref(m), sv, len(s_values), et, ctypes.byref(ki)))
    return list(et), ki.value


def knee_search_table(batch, table, total=TOTAL_SLOTS, start_slots=10, overprov_slots=2):
    """Knee search over the slot counts of a {slots: latency_us} table (host only)."""
    cand = sorted(table)
    sl = (_i * len(cand))(*cand)
    lat = (ctypes.c_int64 * len(cand))(*[table[s] for s in cand])
    r = KneeSearchResult()
    _check(lib().dstack_knee_search_table(batch, sl, lat, len(cand), start_slots, total, overprov_slots,
                                          ctypes.byref(r)))
    return _search_dict(r)


def generate_params(arch, seed, idx):
    """Host-only generation of one weight tensor (bf16 bits, logical layout)."""
    n = ctypes.c_int64()
    _check(lib().dstack_generate_params(arch.encode(), ctypes.c_uint64(seed), idx, None, 0, ctypes.byref(n)))
    out = np.empty(n.value, dtype=np.uint16)
    _check(lib().dstack_generate_params(arch.encode(), ctypes.c_uint64(seed), idx, out.ctypes.data, out.nbytes,
                                        ctypes.byref(n)))
    return out


def _sched_models(models):
    arr = (SchedModel * len(models))()
    for i, m in enumerate(models):
        e = arr[i]
        e.slo_us = m["slo_us"]
        e.max_batch = m["max_batch"]
        e.rate_per_s = m.get("rate_per_s", 0)
        batches = sorted(m["table"])
        slots = sorted({s for b in batches for s in m["table"][b]})
        e.n_batches = len(batches)
        e.n_slots = len(slots)
        for q, b in enumerate(batches):
            e.batches[q] = b
            for r, s in enumerate(slots):
                e.latency_us[q][r] = m["table"][b].get(s, 0)
        for r, s in enumerate(slots):
            e.slots[r] = s
    return arr


def _stats(out):
    return [dict((f, getattr(out.models[i], f)) for f, _ in ModelStats._fields_) for i in range(out.n_models)]


PLACEMENTS = {"lowest": 0, "home": 1}


POLICIES = {"dstack": 0, "maxthroughput": 1, "maxmin": 2, "temporal": 3}


def _sim_params(duration_us, arrivals, fod, sessions_window, policy="dstack", slice_cycle_us=0, resize_violations=0):
    """SimParams plus the arrival buffers it points into (keep them alive)."""
    sp = SimParams()
    sp.duration_us = duration_us
    sp.fod = int(fod)
    sp.sessions_window = sessions_window
    sp.policy = POLICIES[policy]
    sp.slice_cycle_us = slice_cycle_us
    sp.resize_violations = resize_violations
    keep = []
    for i, a in enumerate(arrivals):
        buf = (ctypes.c_int64 * max(1, len(a)))(*a)
        keep.append(buf)
        sp.arrivals_us[i] = ctypes.cast(buf, ctypes.POINTER(ctypes.c_int64))
        sp.n_arrivals[i] = len(a)
    return sp, keep


def simulate(models, period_us, duration_us, arrivals, total_slots=TOTAL_SLOTS, overprov_slots=2, fod=True,
             sessions_window=10, placement="lowest", policy="dstack", slice_cycle_us=0, resize_violations=0):
    """Launcher simulation on the timing table (see dstack_simulate); policy
    "dstack", "maxthroughput", "maxmin" or "temporal".  arrivals: per model
    sorted integer-us arrival times.  Returns a dict."""
    arr = _sched_models(models)
    sp, keep = _sim_params(duration_us, arrivals, fod, sessions_window, policy, slice_cycle_us, resize_violations)
    out = RunOut()
    prm = SchedParams(period_us, total_slots, overprov_slots, PLACEMENTS[placement])
    _check(lib().dstack_simulate(arr, len(models), ctypes.byref(prm), ctypes.byref(sp), ctypes.byref(out)))
    return dict(models=_stats(out), utilisation_ppm=out.utilisation_ppm, job_hash=out.job_hash,
                last_end_us=out.last_end_us)


def simulate_ideal(models, horizon_us, slot_us, total_slots=TOTAL_SLOTS):
    """The ideal slotted, preemptive, kernel-granularity schedule (see
    dstack_simulate_ideal).  models: dicts with per-kernel "slots" and "dur"
    lists, "batch" and "slo_us"."""
    n = len(models)
    keep = []
    arr = (IdealModel * n)()
    for i, m in enumerate(models):
        sl = (_i * len(m["slots"]))(*m["slots"])
        du = (ctypes.c_int64 * len(m["dur"]))(*m["dur"])
        keep += [sl, du]
        arr[i] = IdealModel(len(m["dur"]), m["batch"], sl, du, m["slo_us"])
    out = IdealOut()
    _check(lib().dstack_simulate_ideal(arr, n, horizon_us, slot_us, total_slots, ctypes.byref(out)))
    return dict(items=list(out.items[:n]), forwards=list(out.forwards[:n]), late=list(out.late[:n]),
                busy_slot_us=list(out.busy_slot_us[:n]), utilisation_ppm=out.utilisation_ppm, hash=out.hash)


def serve(handles, tables, inputs, outputs, period_us, duration_us, arrivals, total_slots=TOTAL_SLOTS,
          overprov_slots=2, fod=True, sessions_window=10, log_capacity=1 << 16, policy="dstack", slice_cycle_us=0,
          event_capacity=0, resize_violations=0):
    """Live launcher (see dstack_serve): handles are Model objects, tables the
    timing tables in the form simulate() takes, inputs/outputs device tensors
    sized for each model's max batch; policy "dstack" or "temporal".  Blocks
    for about duration_us.  With event_capacity > 0 the result holds the
    launcher's triggers ("events") for a replay."""
    n = len(handles)
    arr = _sched_models(tables)
    sp, keep = _sim_params(duration_us, arrivals, fod, sessions_window, policy, slice_cycle_us, resize_violations)
    hv = (_vp * n)(*[m.h.value for m in handles])
    iv = (_vp * n)(*[t.data_ptr() for t in inputs])
    ov = (_vp * n)(*[t.data_ptr() for t in outputs])
    prm = SchedParams(period_us, total_slots, overprov_slots, PLACEMENTS["home"])
    out = RunOut()
    log = (JobRecord * max(1, log_capacity))()
    n_log = ctypes.c_int(0)
    evs = (ServeEvent * max(1, event_capacity))()
    n_ev = ctypes.c_int(0)
    _check(lib().dstack_serve(hv, n, iv, ov, arr, ctypes.byref(prm), ctypes.byref(sp), ctypes.byref(out), log,
                              log_capacity, ctypes.byref(n_log), evs, event_capacity, ctypes.byref(n_ev)))
    jobs = [dict((f, getattr(r, f)) for f, _ in JobRecord._fields_) for r in log[:min(n_log.value, log_capacity)]]
    events = [dict((f, getattr(r, f)) for f, _ in ServeEvent._fields_) for r in evs[:min(n_ev.value, event_capacity)]]
    return dict(models=_stats(out), utilisation_ppm=out.utilisation_ppm, job_hash=out.job_hash,
                last_end_us=out.last_end_us, n_jobs=n_log.value, log=jobs, n_events=n_ev.value, events=events)


def schedule(models, period_us, total_slots=TOTAL_SLOTS, overprov_slots=2, placement="lowest"):
    """models: list of dicts {slo_us, max_batch, rate_per_s, table: {batch: {slots: latency_us}}}.
    Returns (status, result dict); status is OK or E_INFEASIBLE (plan still filled)."""
    arr = (SchedModel * len(models))()
    for i, m in enumerate(models):
        e = arr[i]
        e.slo_us = m["slo_us"]
        e.max_batch = m["max_batch"]
        e.rate_per_s = m.get("rate_per_s", 0)
        batches = sorted(m["table"])
        slots = sorted({s for b in batches for s in m["table"][b]})
        e.n_batches = len(batches)
        e.n_slots = len(slots)
        for q, b in enumerate(batches):
            e.batches[q] = b
            for r, s in enumerate(slots):
                e.latency_us[q][r] = m["table"][b].get(s, 0)
        for r, s in enumerate(slots):
            e.slots[r] = s
    prm = SchedParams(period_us, total_slots, overprov_slots, PLACEMENTS[placement])
    out = ScheduleOut()
    st = lib().dstack_schedule(arr, len(models), ctypes.byref(prm), ctypes.byref(out))
    if st not in (OK, E_INFEASIBLE):
        _check(st)
    n = out.n_models
    jobs = [dict(model=j.model, k=j.k, release=j.release_us, deadline=j.deadline_us, start=j.start_us,
                 duration=j.duration_us, slots=j.slots, missed=j.missed, slot_mask=j.slot_mask)
            for j in out.jobs[:out.n_jobs]]
    return st, dict(batch=list(out.batch[:n]), knee_slots=list(out.knee_slots[:n]),
                    deployed_slots=list(out.deployed_slots[:n]), latency_us=list(out.latency_us[:n]),
                    feasible=list(out.feasible[:n]), jobs=jobs, utilisation_ppm=out.utilisation_ppm,
                    home_offset=list(out.home_offset[:n]) if placement == "home" else None)


# ---------------------------------------------------------- kernel ops ----

def _stream(stream):
    if stream is None:
        return None
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def conv2d(x, w, K, R, S, stride, pad, scale, shift, res, act, y, out_fp32=False, stream=None):
    N, H, W, C = x.shape
    _check(lib().dstack_op_conv2d(_ptr(x), N, H, W, C, _ptr(w), K, R, S, stride, pad, _ptr(scale), _ptr(shift),
                                  _ptr(res), act, _ptr(y), int(out_fp32), _stream(stream)))


def conv2d_ws(x, w, K, R, S, stride, pad, scale, shift, res, act, y, workspace, out_fp32=False, n_cu=0,
              stream=None):
    """conv2d with the depth split; workspace: a 256-byte aligned device
    buffer (torch tensor or None) whose first 16 KiB are zero before its first use."""
    N, H, W, C = x.shape
    wsb = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(lib().dstack_op_conv2d_ws(_ptr(x), N, H, W, C, _ptr(w), K, R, S, stride, pad, _ptr(scale), _ptr(shift),
                                     _ptr(res), act, _ptr(y), int(out_fp32), int(n_cu), _ptr(workspace), wsb,
                                     _stream(stream)))


UNLIMITED = ctypes.c_size_t(-1).value


def conv2d_noalloc(x, w, K, R, S, stride, pad, scale, shift, res, act, y, out_fp32=False, n_cu=0, stream=None):
    """conv2d_ws on the library's fixed split-K scratch (allocates nothing)."""
    N, H, W, C = x.shape
    _check(lib().dstack_op_conv2d_noalloc(_ptr(x), N, H, W, C, _ptr(w), K, R, S, stride, pad, _ptr(scale),
                                          _ptr(shift), _ptr(res), act, _ptr(y), int(out_fp32), int(n_cu),
                                          _stream(stream)))


def conv2d_noalloc_scratch_bytes():
    return lib().dstack_conv2d_noalloc_scratch_bytes()


def conv2d_plan(N, H, W, C, K, R, S, stride, pad, act=0, out_fp32=False, n_cu=0, workspace_bytes=UNLIMITED):
    p = ConvPlan()
    _check(lib().dstack_conv2d_plan(N, H, W, C, K, R, S, stride, pad, act, int(out_fp32), int(n_cu),
                                    workspace_bytes, ctypes.byref(p)))
    return dict((f, getattr(p, f)) for f, _ in ConvPlan._fields_ if f != "pad")


def arch_convs(arch, batch):
    """The implicit-GEMM convolutions of one forward (host only), as dicts of conv2d arguments."""
    n = ctypes.c_int()
    _check(lib().dstack_arch_convs(arch.encode(), batch, None, 0, ctypes.byref(n)))
    out = (ConvShape * n.value)()
    _check(lib().dstack_arch_convs(arch.encode(), batch, out, n.value, ctypes.byref(n)))
    return [dict((f, getattr(c, f)) for f, _ in ConvShape._fields_) for c in out]


def partition_count():
    """(live partitions, the limit)."""
    a, b = ctypes.c_int(), ctypes.c_int()
    _check(lib().dstack_partition_count(ctypes.byref(a), ctypes.byref(b)))
    return a.value, b.value


def conv2d_rgb(x, w4, K, R, stride, pad, scale, shift, act, y, stream=None):
    """x [N,H,W,3] bf16, w4 [K,R,R,4] bf16 (channel 3 zero) -> y [N,Ho,Wo,K] bf16."""
    N, H, W, C = x.shape
    assert C == 3
    _check(lib().dstack_op_conv2d_rgb(_ptr(x), N, H, W, _ptr(w4), K, R, stride, pad, _ptr(scale), _ptr(shift), act,
                                      _ptr(y), _stream(stream)))


def expand_dw(x, we, Ce, se, he, act_e, wd_rsc, stride, sd, hd, act_d, y, stream=None):
    """x [N,H,W,Cin] -> act_d(sd * dw3x3(act_e(se * (x @ we^T) + he)) + hd) -> y [N,Ho,Wo,Ce] (bf16)."""
    N, H, W, Cin = x.shape
    _check(lib().dstack_op_expand_dw(_ptr(x), N, H, W, Cin, _ptr(we), Ce, _ptr(se), _ptr(he), act_e, _ptr(wd_rsc),
                                     stride, _ptr(sd), _ptr(hd), act_d, _ptr(y), _stream(stream)))


def dwconv3x3(x, w_rsc, stride, scale, shift, act, y, stream=None):
    N, H, W, C = x.shape
    _check(lib().dstack_op_dwconv3x3(_ptr(x), N, H, W, C, _ptr(w_rsc), stride, _ptr(scale), _ptr(shift), act,
                                     _ptr(y), _stream(stream)))


def fc_workspace_bytes(B, I, O):
    return lib().dstack_fc_workspace_bytes(B, I, O)


def fc(x, w, bias, act, y, out_fp32=False, workspace=None, stream=None):
    """workspace: optional device buffer for the depth split's partial sums."""
    B, I = x.shape
    O = w.shape[0]
    wsb = workspace.numel() * workspace.element_size() if workspace is not None else 0
    _check(lib().dstack_op_fc(_ptr(x), B, I, _ptr(w), _ptr(bias), O, act, _ptr(y), int(out_fp32), _ptr(workspace),
                              wsb, _stream(stream)))


def maxpool(x, k, stride, pad, y, stream=None):
    N, H, W, C = x.shape
    _check(lib().dstack_op_maxpool(_ptr(x), N, H, W, C, k, stride, pad, _ptr(y), _stream(stream)))


def avgpool(x, y, stream=None):
    N, H, W, C = x.shape
    _check(lib().dstack_op_avgpool(_ptr(x), N, H, W, C, _ptr(y), _stream(stream)))


def lstm_workspace_bytes(T, B, H):
    return lib().dstack_lstm_workspace_bytes(T, B, H)


def lstm_layer(x, w_ih, w_hh, bias, h_bf16, h_f32, workspace, stream=None):
    T, B, I = x.shape
    H = w_hh.shape[1]
    _check(lib().dstack_op_lstm_layer(_ptr(x), T, B, I, H, _ptr(w_ih), _ptr(w_hh), _ptr(bias), _ptr(h_bf16),
                                      _ptr(h_f32), _ptr(workspace), _stream(stream)))


def embed_ln(ids, T, we, pe, te, gamma, beta, eps, y, stream=None):
    """ids [rows] int32 -> y [rows,H] bf16 (see dstack_op_embed_ln)."""
    vocab, H = we.shape
    _check(lib().dstack_op_embed_ln(_ptr(ids), ids.numel(), T, vocab, _ptr(we), _ptr(pe), _ptr(te), H, _ptr(gamma),
                                    _ptr(beta), float(eps), _ptr(y), _stream(stream)))


def layernorm(x, gamma, beta, eps, y, stream=None):
    """x [rows,H] bf16 -> y bf16 (see dstack_op_layernorm)."""
    H = x.shape[-1]
    _check(lib().dstack_op_layernorm(_ptr(x), x.numel() // H, H, _ptr(gamma), _ptr(beta), float(eps), _ptr(y),
                                     _stream(stream)))


def attention(qkv, heads, out, stream=None):
    """qkv [B,T,3*heads*dh] bf16 -> out [B,T,heads*dh] bf16 (see dstack_op_attention)."""
    B, T, H3 = qkv.shape
    _check(lib().dstack_op_attention(_ptr(qkv), B, T, heads, H3 // 3 // heads, _ptr(out), _stream(stream)))

