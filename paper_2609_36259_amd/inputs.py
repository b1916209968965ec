"""Seeded synthetic workloads for the CyFA core operator.

This module is shared by the tests, the benchmark and the oracle harness.  It
holds only the input recipe (distributions, draw order, rounding of the inputs
to the storage dtype) and none of the operator's arithmetic.

Recipe (one ``numpy.random.Generator(PCG64(seed))`` per workload, draws in this
order): q, k ~ N(0,1) then L2-normalised per (token, head) vector; v ~ N(0,1);
clock increment delta = softplus(N(mu_delta, 1)); forget log-gate
g = log alpha = logsigmoid(N(3, 1)); write strength beta = sigmoid(N(0, 1));
readout R_h = I + 0.1 N(0, 1).  beta and R are drawn after the tensors the
workloads name, so the named tensors do not depend on whether they are used.
bf16 workloads round q, k, v to bf16 (round to nearest even) once; both the
GPU and the oracle consume exactly those rounded values.

The shapes stand in for the paper's 400M-1.4B language-model layers (Sec. 4.1
and the model configuration table of App. C); the paper's training corpus and
evaluation suites are not used.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

M_ACTIVE = 127          # active relative-time slots (Sec. 3.4)
M_STORAGE = 128         # storage rows, the last one is padding (App. A.7)


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    T: int
    H: int
    dk: int
    dv: int
    chunk: int = 64
    seed: int = 0
    dtype: str = "bf16"          # storage dtype of q, k, v, o: "f32" | "bf16"
    delta_mu: float = 0.0        # mean of the normal fed to softplus for delta
    m: int = M_ACTIVE
    extra: dict = field(default_factory=dict, compare=False, hash=False)

    @property
    def tokens(self) -> int:
        return self.B * self.T

    @property
    def token_heads(self) -> int:
        return self.B * self.T * self.H


# The five workloads: tiny fp32 forward, 400M-scale layer, 1.4B-scale layer
# (headline), long-context slow-clock forward, and the recurrent decode step.
FWD_TINY = Workload("tiny-f32 B1 T256 H2 d64", 1, 256, 2, 64, 64, seed=0, dtype="f32")
FWD_400M = Workload("400M-layer B8 T2048 H8 d128", 8, 2048, 8, 128, 128, seed=1)
FWD_1P4B = Workload("1.4B-layer B4 T4096 H16 d128", 4, 4096, 16, 128, 128, seed=2)
FWD_LONG = Workload("long-ctx B1 T32768 H16 d128 slow-clock", 1, 32768, 16, 128, 128,
                    seed=3, delta_mu=-1.0)
DECODE = Workload("decode N256 H16 d128 prefix512 steps64", 256, 512 + 64, 16, 128, 128,
                  seed=4, dtype="f32", extra={"prefix": 512, "steps": 64})
# The paper's own operator benchmark shape (its 400M model's layer at 2K tokens:
# 4 heads of 256 channels, 32 sequences), with the value distributions above.
FWD_PAPER_OP = Workload("paper-op B32 T2048 H4 d256", 32, 2048, 4, 256, 256, seed=5)
# The largest slot count of the paper's ablation (m = 255, 256 storage rows) at the
# 1.4B-scale layer shape.
FWD_1P4B_M255 = Workload("1.4B-layer m255 B4 T4096 H16 d128", 4, 4096, 16, 128, 128, seed=6, m=255)
# the smallest slot count of the same ablation (m = 63) at the same layer shape
FWD_1P4B_M63 = Workload("1.4B-layer m63 B4 T4096 H16 d128", 4, 4096, 16, 128, 128, seed=7, m=63)

FORWARD_WORKLOADS = (FWD_TINY, FWD_400M, FWD_1P4B, FWD_LONG)


def round_bf16(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 (ties to even); returns float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16 << 16
    return u.astype(np.uint32).view(np.float32)


def _softplus(x):
    return np.logaddexp(0.0, x)


def _logsigmoid(x):
    return -np.logaddexp(0.0, -x)


def _sigmoid(x):
    return 0.5 * (1.0 + np.tanh(0.5 * x))


def _unit_rows(x):
    n = np.sqrt(np.sum(x.astype(np.float64) ** 2, axis=-1, keepdims=True))
    return (x / np.maximum(n, 1e-30)).astype(np.float32)


def draw_sequence_tensors(rng: np.random.Generator, lead: tuple, H: int, dk: int, dv: int,
                          delta_mu: float, dtype: str):
    """Draw q, k, v, delta, g, beta_raw for an array of shape ``lead + (H, ...)``."""
    q = _unit_rows(rng.standard_normal(lead + (H, dk), dtype=np.float32))
    k = _unit_rows(rng.standard_normal(lead + (H, dk), dtype=np.float32))
    v = rng.standard_normal(lead + (H, dv), dtype=np.float32)
    delta = _softplus(rng.standard_normal(lead + (H,)) + delta_mu).astype(np.float32)
    g = _logsigmoid(rng.standard_normal(lead + (H,)) + 3.0).astype(np.float32)
    beta = _sigmoid(rng.standard_normal(lead + (H,))).astype(np.float32)
    if dtype == "bf16":
        q, k, v = round_bf16(q), round_bf16(k), round_bf16(v)
    elif dtype != "f32":
        raise ValueError(f"unknown dtype {dtype!r}")
    return q, k, v, delta, g, beta


def draw_readout(rng: np.random.Generator, H: int, m: int) -> np.ndarray:
    return (np.eye(m, dtype=np.float64)[None] +
            0.1 * rng.standard_normal((H, m, m))).astype(np.float32)


def make_forward_inputs(B: int, T: int, H: int, dk: int, dv: int, seed: int,
                        dtype: str = "bf16", delta_mu: float = 0.0, m: int = M_ACTIVE,
                        with_beta: bool = True, with_R: bool = True) -> dict:
    """Seeded forward inputs with layout q,k:[B,T,H,dk] v:[B,T,H,dv] scalars:[B,T,H].

    Returns float32 numpy arrays (q, k, v already rounded when dtype is bf16),
    ``beta``/``R`` set to None when not requested, and the default logit scale
    dk**-0.5.
    """
    rng = np.random.Generator(np.random.PCG64(seed))
    q, k, v, delta, g, beta = draw_sequence_tensors(rng, (B, T), H, dk, dv, delta_mu, dtype)
    R = draw_readout(rng, H, m)
    return dict(q=q, k=k, v=v, delta=delta, log_alpha=g,
                beta=beta if with_beta else None, R=R if with_R else None,
                scale=float(dk) ** -0.5, m=m, dtype=dtype)


def workload_inputs(w: Workload, **kw) -> dict:
    return make_forward_inputs(w.B, w.T, w.H, w.dk, w.dv, w.seed, w.dtype, w.delta_mu,
                               w.m, **kw)


def make_decode_inputs(N: int, H: int, d: int, prefix: int, steps: int, seed: int,
                       streams=None, m: int = M_ACTIVE) -> dict:
    """Per-stream seeded decode inputs: stream n draws its own prefix+steps tokens.

    Stream n uses ``SeedSequence(seed).spawn(N)[n]``, so any subset of streams can
    be regenerated alone.  Arrays are laid out [len(streams), prefix+steps, H, ...].
    R comes from a separate child of the same seed sequence.
    """
    ss = np.random.SeedSequence(seed)
    children = ss.spawn(N + 1)
    streams = list(range(N)) if streams is None else list(streams)
    L = prefix + steps
    out = {key: [] for key in ("q", "k", "v", "delta", "log_alpha", "beta")}
    for n in streams:
        rng = np.random.Generator(np.random.PCG64(children[n]))
        q, k, v, delta, g, beta = draw_sequence_tensors(rng, (L,), H, d, d, 0.0, "f32")
        for key, val in zip(out, (q, k, v, delta, g, beta)):
            out[key].append(val)
    res = {key: np.stack(val) for key, val in out.items()}
    res["R"] = draw_readout(np.random.Generator(np.random.PCG64(children[N])), H, m)
    res.update(scale=float(d) ** -0.5, m=m, prefix=prefix, steps=steps, streams=streams)
    return res
