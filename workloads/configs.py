"""The five synthetic workloads of the sparse-embedding hot path.

Each workload stands in for one of the paper's NLP training jobs (Sec. 5.2.2:
LM on LM1B, GNMT-8 on WMT-16, Transformer on WMT-14, BERT on SQuAD).  Those
datasets are not used; token ids are seeded Zipf (or uniform) draws with the
shapes below, gradients and weights are seeded normals.

A workload is a list of tables; each table has its own vocabulary V, width D,
tokens per batch T, id law, gradient dtype and sigma, shard count P with a
row-to-owner rule, and a seed.  `make_table_state` / `make_batch` return numpy
arrays; nothing here computes any step of the method.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

from . import gen


@dataclass(frozen=True)
class TableSpec:
    V: int
    D: int
    T: int
    id_law: str              # "zipf" or "uniform"
    zipf_s: float            # exponent when id_law == "zipf"
    grad_dtype: str          # "f32" or "bf16"
    grad_sigma: float
    P: int
    owner_rule: str          # "mod" or "range"
    seed: int


@dataclass(frozen=True)
class Workload:
    name: str
    description: str
    tables: tuple
    steps: int
    lr: float = 1e-3
    beta1: float = 0.9
    beta2: float = 0.999
    eps: float = 1e-8
    extra: dict = field(default_factory=dict)


WORKLOADS = {
    "tiny": Workload(
        "tiny", "V=1000 D=64 fp32, 512 ids Zipf(1.1), P=2 id mod P, one Adam step",
        (TableSpec(1000, 64, 512, "zipf", 1.1, "f32", 1.0, 2, "mod", 1),), steps=1),
    "transformer_shared_vocab": Workload(
        "transformer_shared_vocab",
        "V=32768 D=512 fp32, 25000 ids Zipf(1.0), grads N(0,0.01), P=4 contiguous ranges, 10 steps",
        (TableSpec(32768, 512, 25000, "zipf", 1.0, "f32", 0.01, 4, "range", 2),), steps=10),
    "two_table_translation": Workload(
        "two_table_translation",
        "source+target tables V=32000 D=1024 fp32, 16384 ids each Zipf(1.05), P=8 id mod P",
        (TableSpec(32000, 1024, 16384, "zipf", 1.05, "f32", 0.01, 8, "mod", 31),
         TableSpec(32000, 1024, 16384, "zipf", 1.05, "f32", 0.01, 8, "mod", 32)), steps=3),
    "lm_large_vocab_bf16": Workload(
        "lm_large_vocab_bf16",
        "V=262144 D=1024 fp32 weights, bf16 grads N(0,0.01), 16384 ids Zipf(1.0), P=8 contiguous ranges",
        (TableSpec(262144, 1024, 16384, "zipf", 1.0, "bf16", 0.01, 8, "range", 4),), steps=3),
    "lowdup_uniform": Workload(
        "lowdup_uniform",
        "V=1048576 D=256 fp32, 65536 ids uniform (few repeats), P=16 id mod P",
        (TableSpec(1 << 20, 256, 65536, "uniform", 0.0, "f32", 0.01, 16, "mod", 51),), steps=3),
    "lowdup_zipf13": Workload(
        "lowdup_zipf13",
        "V=1048576 D=256 fp32, 65536 ids Zipf(1.3) (hot rows), P=16 id mod P",
        (TableSpec(1 << 20, 256, 65536, "zipf", 1.3, "f32", 0.01, 16, "mod", 52),), steps=3),
}


def row_owner(spec: TableSpec) -> np.ndarray:
    return gen.owner_mod(spec.V, spec.P) if spec.owner_rule == "mod" else gen.owner_range(spec.V, spec.P)


def make_weights(spec: TableSpec) -> np.ndarray:
    """Initial table, N(0, 1) fp32, shape [V, D]."""
    key = gen.stream_key(spec.seed, 0, gen.PURPOSE_WEIGHTS)
    return gen.normal_f32(key, spec.V * spec.D, 1.0).reshape(spec.V, spec.D)


def make_ids(spec: TableSpec, step: int, T: int | None = None) -> np.ndarray:
    T = spec.T if T is None else T
    key = gen.stream_key(spec.seed, step, gen.PURPOSE_IDS)
    if spec.id_law == "uniform":
        return gen.uniform_ids(key, T, spec.V)
    return gen.zipf_ids(key, T, spec.V, spec.zipf_s)


def make_grads(spec: TableSpec, step: int, T: int | None = None) -> np.ndarray:
    """Per-token gradient rows [T, D]: fp32 array, or uint16 bf16 bit patterns."""
    T = spec.T if T is None else T
    key = gen.stream_key(spec.seed, step, gen.PURPOSE_GRADS)
    g = gen.normal_f32(key, T * spec.D, spec.grad_sigma).reshape(T, spec.D)
    if spec.grad_dtype == "bf16":
        return gen.bf16_round(g).reshape(T, spec.D)
    return g


def make_batch(spec: TableSpec, step: int, T: int | None = None):
    """(ids [T] int32, grads [T, D]) for one training step of one table."""
    return make_ids(spec, step, T), make_grads(spec, step, T)
