"""Seeded synthetic inputs for FAVOR attention (shared by tests and the bench).

This module holds no arithmetic of the method: it only draws Q, K, V (and the
protein-shaped embedding/projection that stands in for a model's attention
inputs) with numpy's seeded generator and rounds them to the storage dtype.
The random features W, b are NOT drawn here: they come from the ORF draw
(library or oracle), whose generator is defined in the library header.

Workloads (d = 64 everywhere):
  bidir_small     B1 H1 L1024  M128 bidirectional, fp32
  bidir_b8h8      B8 H8 L4096  M256 bidirectional, bf16
  causal_b8h8     B8 H8 L8192  M256 unidirectional, bf16
  protein_b4h8    B4 H8 L8192  M256 both directions, bf16; token ids over a
                  25-symbol alphabet embedded to d_model 512 by an N(0, 1/512)
                  table and projected by N(0, 1) W_q, W_k, W_v to 8 heads of 64
                  (stands in for the paper's concatenated-protein task of
                  Sec. 4.4: L = 8192, 25 symbols; no dataset item is used)
  causal_long     B1 H16 L65536 M256 unidirectional, bf16, ORF redrawn per call
Q and K are N(0, 1) scaled by d^-1/4 (protein: after projection); V is N(0, 1).
The library is then run with input_scale = d^-1/4, i.e. it evaluates the
paper's exp(Q K^T / sqrt d) on exactly these tensors.
"""
from dataclasses import dataclass, replace

import numpy as np


def bf16_bits(a):
    """Round float32 values to bfloat16 (round to nearest, ties to even); raw bits."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    r = (u + np.uint64(0x7FFF) + ((u >> np.uint64(16)) & np.uint64(1))) >> np.uint64(16)
    return r.astype(np.uint16)


def bf16_to_f32(bits):
    return (np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_round(a):
    """float32 array holding the bf16-rounded values of a."""
    return bf16_to_f32(bf16_bits(a))


@dataclass(frozen=True)
class Workload:
    name: str
    direction: str        # "bidir", "causal" or "both"
    B: int
    H: int
    L: int
    d: int
    M: int
    dtype: str            # "f32" or "bf16"
    seed: int
    redraw: bool = False  # ORF drawn inside every call
    protein: bool = False

    @property
    def input_scale(self):
        return float(self.d) ** -0.25

    def with_(self, **kw):
        return replace(self, **kw)


WORKLOADS = {
    "bidir_small": Workload("bidir_small", "bidir", 1, 1, 1024, 64, 128, "f32", seed=1),
    "bidir_b8h8": Workload("bidir_b8h8", "bidir", 8, 8, 4096, 64, 256, "bf16", seed=2),
    "causal_b8h8": Workload("causal_b8h8", "causal", 8, 8, 8192, 64, 256, "bf16", seed=3),
    "protein_b4h8": Workload("protein_b4h8", "both", 4, 8, 8192, 64, 256, "bf16", seed=4,
                             protein=True),
    "causal_long": Workload("causal_long", "causal", 1, 16, 65536, 64, 256, "bf16", seed=5,
                            redraw=True),
}

PROTEIN_ALPHABET = 25
PROTEIN_DMODEL = 512


def _round(x, dtype):
    x = np.asarray(x, dtype=np.float32)
    return bf16_round(x) if dtype == "bf16" else x


def make_qkv(w, seed=None):
    """Q, K, V as float32 arrays [B, H, L, d] holding values exact in w.dtype."""
    seed = w.seed if seed is None else seed
    rng = np.random.default_rng(seed)
    B, H, L, d = w.B, w.H, w.L, w.d
    qk_scale = np.float32(float(d) ** -0.25)
    if not w.protein:
        Q = rng.standard_normal((B, H, L, d), dtype=np.float32) * qk_scale
        K = rng.standard_normal((B, H, L, d), dtype=np.float32) * qk_scale
        V = rng.standard_normal((B, H, L, d), dtype=np.float32)
    else:
        dm = PROTEIN_DMODEL
        assert H * d == dm, "protein workload projects d_model onto H heads of d"
        ids = rng.integers(0, PROTEIN_ALPHABET, size=(B, L))
        emb = rng.standard_normal((PROTEIN_ALPHABET, dm)) / np.sqrt(dm)
        Wq, Wk, Wv = (rng.standard_normal((dm, dm)) for _ in range(3))
        # only 25 distinct embedding rows exist, so project the table, then gather
        def heads(Wp):
            table = (emb @ Wp).astype(np.float32)            # [25, 512]
            x = table[ids]                                   # [B, L, 512]
            return np.ascontiguousarray(x.reshape(B, L, H, d).transpose(0, 2, 1, 3))
        Q = heads(Wq) * qk_scale
        K = heads(Wk) * qk_scale
        V = heads(Wv)
    return _round(Q, w.dtype), _round(K, w.dtype), _round(V, w.dtype)


def protein_ids(w, seed=None):
    """Token ids of the protein workload (same draw order as make_qkv)."""
    seed = w.seed if seed is None else seed
    rng = np.random.default_rng(seed)
    return rng.integers(0, PROTEIN_ALPHABET, size=(w.B, w.L))
