"""Oracle for the D-STACK hot path (arxiv 2304.13541).

TEST INFRASTRUCTURE ONLY.  Only ``tests/``, ``__graft_entry__.smoke()`` and
the CPU-baseline leg of ``bench.py`` may import this package.  It shares no
code with the HIP library and never imports it.

* ``oracle_numerics.c`` -- fp64 forward passes (direct convolution, naive
  products, LSTM, layer norm and attention for the BERT encoder), built here
  with gcc into ``liboracle.so``.
* ``sched.py`` -- the scheduling decisions (knee, SLO-constrained batch
  optimisation, spatio-temporal session plan, utilisation) in integer Python.
* ``knee_model.py`` -- the analytical DNN latency model of Sec. 4.3 and its
  knee in plain fp64 Python.
"""
import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle_numerics.c")
# ORACLE_LIBRARY may name the CPU sanitizer build (liboracle_san.so, see build()).
_LIB = os.environ.get("ORACLE_LIBRARY") or os.path.join(_HERE, "liboracle.so")
_SAN_LIB = os.path.join(_HERE, "liboracle_san.so")
_lib = None


def build(force=False, sanitize=False):
    """Compile the fp64 numerics with gcc (no GPU involved).  sanitize=True
    builds liboracle_san.so with clang's AddressSanitizer and
    UndefinedBehaviorSanitizer instead (the runtime the library's sanitizer
    build uses, so both load into one process)."""
    if sanitize:
        tmp = _SAN_LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["/opt/rocm/llvm/bin/clang", "-O1", "-g", "-fopenmp", "-ffp-contract=off", "-shared",
                               "-fPIC", "-fsanitize=address,undefined", "-fno-sanitize-recover=undefined",
                               "-fno-omit-frame-pointer", "-shared-libasan", "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _SAN_LIB)
        return _SAN_LIB
    if os.environ.get("ORACLE_LIBRARY"):  # a prebuilt variant was named: use it as it is
        return _LIB
    if force or not os.path.exists(_LIB) or os.path.getmtime(_LIB) < os.path.getmtime(_SRC):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(["gcc", "-O2", "-fopenmp", "-ffp-contract=off", "-shared", "-fPIC",
                               "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, _LIB)
    return _LIB


def lib():
    global _lib
    if _lib is None:
        build()
        L = ctypes.CDLL(_LIB)
        dp = ctypes.POINTER(ctypes.c_double)
        L.oracle_bf16_round.restype = ctypes.c_double
        L.oracle_bf16_round.argtypes = [ctypes.c_double]
        L.oracle_bf16_to_double.restype = ctypes.c_double
        L.oracle_bf16_to_double.argtypes = [ctypes.c_uint16]
        L.oracle_model_load.restype = ctypes.c_void_p
        L.oracle_model_load.argtypes = [ctypes.c_char_p, ctypes.c_uint64]
        L.oracle_model_free.argtypes = [ctypes.c_void_p]
        L.oracle_model_num_tensors.argtypes = [ctypes.c_void_p]
        L.oracle_model_tensor_numel.restype = ctypes.c_long
        L.oracle_model_tensor_numel.argtypes = [ctypes.c_void_p, ctypes.c_int]
        L.oracle_model_tensor_bf16.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p]
        L.oracle_model_forward.argtypes = [ctypes.c_void_p, ctypes.c_int, ctypes.c_void_p, ctypes.c_int, dp]
        L.oracle_model_set_tensor.argtypes = [ctypes.c_void_p, ctypes.c_int, dp]
        L.oracle_splitmix64.argtypes = [ctypes.c_uint64, ctypes.c_int, ctypes.c_void_p]
        i = ctypes.c_int
        L.oracle_conv2d.argtypes = [dp, i, i, i, i, dp, i, i, i, i, i, dp]
        L.oracle_dwconv.argtypes = [dp, i, i, i, i, dp, i, i, i, i, dp]
        L.oracle_fc.argtypes = [dp, i, i, dp, dp, i, dp]
        L.oracle_maxpool.argtypes = [dp, i, i, i, i, i, i, i, dp]
        L.oracle_avgpool.argtypes = [dp, i, i, i, i, dp]
        L.oracle_lstm_layer.argtypes = [dp, i, i, i, i, dp, dp, dp, dp, i, dp, dp]
        L.oracle_layernorm.argtypes = [dp, ctypes.c_long, i, dp, dp, ctypes.c_double, dp]
        L.oracle_attention.argtypes = [dp, i, i, i, i, dp]
        L.oracle_bert_forward.argtypes = [ctypes.c_void_p, i, ctypes.c_void_p, i, dp]
        L.oracle_bert_hidden.argtypes = [ctypes.c_void_p, i, ctypes.c_void_p, i, i, dp]
        L.oracle_bert_layer.argtypes = [ctypes.c_void_p, i, i, dp, i, dp]
        _lib = L
    return _lib


def _dp(a):
    return a.ctypes.data_as(ctypes.POINTER(ctypes.c_double))


def _f64(a):
    return np.ascontiguousarray(a, dtype=np.float64)


# ---------------------------------------------------------------- bf16 ----

def bf16_round(x):
    """Round-to-nearest-even to bf16, element-wise, returned as float64."""
    f = lib().oracle_bf16_round
    a = _f64(x)
    return np.vectorize(f, otypes=[np.float64])(a) if a.ndim else np.float64(f(float(a)))


def bf16_bits_to_f64(bits):
    """bf16 bit patterns (uint16) -> exact float64 values."""
    b = np.ascontiguousarray(bits, dtype=np.uint16)
    return (b.astype(np.uint32) << 16).view(np.float32).astype(np.float64)


# ------------------------------------------------------------ layers ----

def out_dim(n, k, stride, pad):
    return (n + 2 * pad - k) // stride + 1


def conv2d(x, w, stride, pad):
    """x [N,H,W,C], w [K,R,S,C] -> y [N,Ho,Wo,K] (fp64 direct cross-correlation)."""
    x, w = _f64(x), _f64(w)
    N, H, W, C = x.shape
    K, R, S, C2 = w.shape
    assert C == C2
    y = np.empty((N, out_dim(H, R, stride, pad), out_dim(W, S, stride, pad), K))
    lib().oracle_conv2d(_dp(x), N, H, W, C, _dp(w), K, R, S, stride, pad, _dp(y))
    return y


def dwconv(x, w, stride, pad):
    """x [N,H,W,C], w [C,R,S] -> y [N,Ho,Wo,C]."""
    x, w = _f64(x), _f64(w)
    N, H, W, C = x.shape
    C2, R, S = w.shape
    assert C == C2
    y = np.empty((N, out_dim(H, R, stride, pad), out_dim(W, S, stride, pad), C))
    lib().oracle_dwconv(_dp(x), N, H, W, C, _dp(w), R, S, stride, pad, _dp(y))
    return y


def fc(x, w, b=None):
    """x [B,I], w [O,I], b [O] -> x w^T + b."""
    x, w = _f64(x), _f64(w)
    B, I = x.shape
    O = w.shape[0]
    y = np.empty((B, O))
    bb = _f64(b) if b is not None else np.zeros(O)
    lib().oracle_fc(_dp(x), B, I, _dp(w), _dp(bb), O, _dp(y))
    return y


def maxpool(x, k, stride, pad):
    x = _f64(x)
    N, H, W, C = x.shape
    y = np.empty((N, out_dim(H, k, stride, pad), out_dim(W, k, stride, pad), C))
    lib().oracle_maxpool(_dp(x), N, H, W, C, k, stride, pad, _dp(y))
    return y


def avgpool(x):
    x = _f64(x)
    N, H, W, C = x.shape
    y = np.empty((N, C))
    lib().oracle_avgpool(_dp(x), N, H, W, C, _dp(y))
    return y


def lstm_layer(x, w_ih, w_hh, b_ih, b_hh, round_h=False):
    """x [T,B,I] -> (h [T,B,H], c_T [B,H]); gate order i, f, g, o."""
    x, w_ih, w_hh, b_ih, b_hh = map(_f64, (x, w_ih, w_hh, b_ih, b_hh))
    T, B, I = x.shape
    Hd = w_hh.shape[1]
    h = np.empty((T, B, Hd))
    c = np.empty((B, Hd))
    lib().oracle_lstm_layer(_dp(x), T, B, I, Hd, _dp(w_ih), _dp(w_hh), _dp(b_ih), _dp(b_hh), int(round_h),
                            _dp(h), _dp(c))
    return h, c


def layernorm(x, gamma, beta, eps):
    """Rows of x [..., C] normalised by their mean and biased variance, then * gamma + beta."""
    x = _f64(x)
    C = x.shape[-1]
    rows = x.size // C
    y = np.empty_like(x)
    lib().oracle_layernorm(_dp(x), rows, C, _dp(_f64(gamma)), _dp(_f64(beta)), float(eps), _dp(y))
    return y


def attention(qkv, heads):
    """qkv [B,T,3*Hm] (queries, keys, values) -> softmax(q k^T / sqrt(dh)) v per head, [B,T,Hm]."""
    qkv = _f64(qkv)
    B, T, H3 = qkv.shape
    Hm = H3 // 3
    out = np.empty((B, T, Hm))
    lib().oracle_attention(_dp(qkv), B, T, heads, Hm // heads, _dp(out))
    return out


# ------------------------------------------------------------ models ----

ARCHS = ("tinycnn", "resnet50", "mobilenetv2", "vgg19", "lstm2", "bert", "bert_long")
NUM_CLASSES = {"tinycnn": 10, "resnet50": 1000, "mobilenetv2": 1000, "vgg19": 1000, "bert": 2, "bert_long": 2}
BERT_TOKENS = {"bert": 20, "bert_long": 40}


class Model:
    """One architecture with weights drawn from ``seed`` by the oracle's own generator."""

    def __init__(self, arch, seed):
        self.arch = arch
        self.h = lib().oracle_model_load(arch.encode(), ctypes.c_uint64(seed))
        if not self.h:
            raise ValueError("unknown arch %r" % arch)

    def __del__(self):
        if getattr(self, "h", None):
            lib().oracle_model_free(self.h)
            self.h = None

    def num_tensors(self):
        return lib().oracle_model_num_tensors(self.h)

    def tensor_bf16(self, i):
        n = lib().oracle_model_tensor_numel(self.h, i)
        out = np.empty(n, dtype=np.uint16)
        assert lib().oracle_model_tensor_bf16(self.h, i, out.ctypes.data) == 0
        return out

    def numel(self, i):
        return lib().oracle_model_tensor_numel(self.h, i)

    def set_tensor(self, i, values):
        """Plant values into tensor i (tests only)."""
        v = _f64(values).ravel()
        assert v.size == self.numel(i)
        assert lib().oracle_model_set_tensor(self.h, i, _dp(v)) == 0

    def forward(self, x_bits, parity=True):
        """x_bits: bf16 bit patterns. CNN [n,H,W,3] -> [n,classes]; LSTM [50,n,512] -> [50,n,1024];
        BERT: int32 token ids [n,T] -> [n,2]."""
        if self.arch in BERT_TOKENS:
            ids = np.ascontiguousarray(x_bits, dtype=np.int32)
            n = ids.shape[0]
            assert ids.shape == (n, BERT_TOKENS[self.arch])
            out = np.empty((n, 2))
            assert lib().oracle_bert_forward(self.h, n, ids.ctypes.data, int(parity), _dp(out)) == 0
            return out
        x_bits = np.ascontiguousarray(x_bits, dtype=np.uint16)
        if self.arch == "lstm2":
            T, n, _ = x_bits.shape
            out = np.empty((T, n, 1024))
        else:
            n = x_bits.shape[0]
            out = np.empty((n, NUM_CLASSES[self.arch]))
        rc = lib().oracle_model_forward(self.h, n, x_bits.ctypes.data, int(parity), _dp(out))
        assert rc == 0
        return out


def bert_hidden(model, ids, parity=True, layers=12):
    """The hidden state [n, T, 768] after encoder layer `layers` (0: the embeddings; 12: the
    encoder's output) of a BERT model for int32 token ids [n, T]."""
    ids = np.ascontiguousarray(ids, dtype=np.int32)
    n, T = ids.shape
    assert T == BERT_TOKENS[model.arch]
    out = np.empty((n, T, 768))
    assert lib().oracle_bert_hidden(model.h, n, ids.ctypes.data, int(parity), layers, _dp(out)) == 0
    return out


def bert_layer(model, layer, x, parity=True):
    """Encoder layer `layer` (1..12) of a BERT model applied to x [n, T, 768]."""
    x = _f64(x)
    out = np.empty_like(x)
    assert lib().oracle_bert_layer(model.h, x.shape[0], layer, _dp(x), int(parity), _dp(out)) == 0
    return out


def splitmix64(state, n):
    out = np.empty(n, dtype=np.uint64)
    lib().oracle_splitmix64(ctypes.c_uint64(state), n, out.ctypes.data)
    return out


def rel_err(got, ref):
    """Infinity-norm relative error max|g - r| / max|r|."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.max(np.abs(ref))
    return float(np.max(np.abs(got - ref)) / den) if den > 0 else float(np.max(np.abs(got - ref)))
