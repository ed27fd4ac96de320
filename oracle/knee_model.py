"""Analytical DNN latency model and its knee (Sec. 4.3), plain fp64 Python.

TEST INFRASTRUCTURE ONLY (see the package docstring).  This is the slow,
literal statement of the model the library's ``dstack_knee_model_*`` calls
must reproduce exactly (same operations in the same order, so the fp64
results are equal bit for bit).

The model (Sec. 4.3):
* Eq. layer_num_ops: the parallelizable operations of kernel i are
  N_1 = p*b and N_i = floor(N_{i-1} - p*b/Kmax) for i >= 2;
* W_i = N_i * t_p (the kernel's parallel work);
* Eq. execution_time_per_layer: E_i = W_i / max(1, min(S, N_i)) on S SMs;
* Eq. memory_latency: the kernel's wait for its data d_i;
* Eq. total_non_paralleizable_time: W_se = b * sum_i R_i * (t_np + E_m,i);
* Eq. total_time_shrinking_kernel: E_t = W_se + sum_i R_i * E_i;
* Eq. first_order_derivative: the most efficient S maximises the magnitude
  1 / (E_t^2 * S).

Readings (each restated in the design notes):
* N_i is clamped at 0 once the decrement reaches it (the text says the work
  falls to about 0 at the last kernel); such a kernel keeps its serialized
  time t_np and has E_i = 0;
* Eq. memory_latency is read as E_m = d_i / (M * S), M being the bandwidth
  per SM: the text states that the total bandwidth grows in proportion to
  the SMs, while the printed d_i * S / M would grow with S (and is not a
  time);
* t_p may differ per kernel (the build's calibrated kernels); the paper's
  own simulation uses one value for all kernels;
* the knee is the first S of the candidate list with the largest
  1 / (E_t^2 * S), compared as E_t^2 * S < best (ties keep the smaller S
  when the list is ascending).
"""
import math
from typing import List, Optional, Sequence


def sequence(p: int, b: int, kmax: int) -> List[float]:
    """N_1..N_Kmax of Eq. layer_num_ops, clamped at 0."""
    if kmax < 1:
        return []
    step = p * b / kmax
    n = [float(p * b)]
    for _ in range(2, kmax + 1):
        n.append(float(max(0, math.floor(n[-1] - step))))
    return n


def kernel_time(n_par: float, t_p: float, s: int) -> float:
    """E_i = W_i / max(1, min(S, N_i)) with W_i = N_i * t_p."""
    w = n_par * t_p
    return w / max(1.0, min(float(s), n_par))


def memory_time(d: float, m: float, s: int) -> float:
    """E_m = d_i / (M * S) (see the readings); no term when M <= 0."""
    if m <= 0.0:
        return 0.0
    return d / (m * float(s))


def total_time(n_par: Sequence[float], t_p: Sequence[float], s: int, t_np: float, b_serial: float = 1.0,
               reps: Optional[Sequence[float]] = None, data: Optional[Sequence[float]] = None,
               m: float = 0.0) -> float:
    """E_t = W_se + sum_i R_i * E_i on S SMs, kernels summed in order."""
    k = len(n_par)
    w_se = 0.0
    for i in range(k):
        r = 1.0 if reps is None else reps[i]
        em = 0.0 if data is None else memory_time(data[i], m, s)
        w_se += r * (t_np + em)
    w_se *= b_serial
    par = 0.0
    for i in range(k):
        r = 1.0 if reps is None else reps[i]
        par += r * kernel_time(n_par[i], t_p[i], s)
    return w_se + par


def knee(n_par, t_p, s_values, t_np, b_serial=1.0, reps=None, data=None, m=0.0):
    """(E_t per candidate S, index of the knee)."""
    et = [total_time(n_par, t_p, s, t_np, b_serial, reps, data, m) for s in s_values]
    best, arg = None, -1
    for j, s in enumerate(s_values):
        v = et[j] * et[j] * float(s)
        if best is None or v < best:
            best, arg = v, j
    return et, arg
