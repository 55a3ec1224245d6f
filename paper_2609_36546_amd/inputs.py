"""Seeded synthetic workloads for verifier-side window scoring.

This module holds the shapes of the five benchmark workloads and seeded
generators for their raw inputs: query rows, the window's new keys and
values, paged KV pools with their page tables, context lengths, window
lengths, drivers, LM-head hidden rows and weights, and the per-row uniforms
a synthetic proposer draws.  It holds none of the scoring arithmetic
(attention, log-softmax, top-K, the accept rule); both the HIP path and the
CPU oracle consume what it produces.

Workload recipe (stands in for the paper's Qwen3 / DAPO-Math rollouts, whose
data and weights are not used):

* context lengths are integers drawn uniformly (inclusive) per sequence;
* window lengths are fixed per workload or drawn from {1, 4, 8, 16};
* queries, window keys/values and cached keys/values are N(0, 1);
* hidden rows are N(0, 1) divided by their own RMS; LM-head weights are
  N(0, 0.02^2);
* floating-point values are drawn in fp32 and rounded to the storage dtype
  with torch's round-to-nearest-even conversion;
* pages of every sequence come from a seeded permutation of the pool; page
  table entries past a sequence's need, and every slot that holds no cached
  or appended token, point at / hold poison (NaN) when ``poison=True``.

KV pool layouts (the library's documented layouts):

* ``k_pool[num_pages, Hkv, D/32, page_size, 32]`` -- a page holds, per KV
  head and per 32-channel slice, its tokens' 32 key channels one after another
  (key channel d of a slot is at [.., d // 32, slot, d % 32]);
* ``v_pool[num_pages, Hkv, D, page_size]`` -- a page holds, per KV head and
  per channel, the values of its tokens one after another (channel-major).
"""
from __future__ import annotations

import dataclasses
from dataclasses import dataclass, field
from typing import List, Optional, Sequence

import numpy as np
import torch

INT32_MAX = 2**31 - 1


@dataclass(frozen=True)
class ModelShape:
    """One verifier model's attention-layer and LM-head shape."""

    name: str
    Hq: int
    Hkv: int
    D: int
    hidden: int
    vocab: int


@dataclass(frozen=True)
class WorkloadConfig:
    """A verify-step workload: batch, shapes, lengths and proposal recipe."""

    id: int                         # seed-stream id of the workload
    name: str
    dtype: str                      # "f32" or "bf16": storage/compute input type
    B: int
    models: Sequence[ModelShape]    # one model, or (student, teacher)
    page_size: int
    k_choices: Sequence[int]        # one value = fixed window length
    ctx_lo: int
    ctx_hi: int
    driver_rule: str                # "alt" | "S" | "T" | "split64"
    p_argmax: float                 # prob. that a proposal is the verifier argmax
    alt_mode: str                   # "uniform" | "softmax"
    alt_temperature: float = 1.0
    K: int = 16
    pool_tokens: Optional[int] = None   # None: twice what the batch needs
    w_std: float = 0.02


STUDENT = ModelShape("qwen3-1.7b-like", Hq=16, Hkv=8, D=128, hidden=2048, vocab=151936)
TEACHER = ModelShape("qwen3-30b-a3b-like", Hq=32, Hkv=4, D=128, hidden=2048, vocab=151936)
TINY = ModelShape("tiny", Hq=4, Hkv=2, D=64, hidden=256, vocab=1024)

WORKLOADS = {
    "tiny-f32": WorkloadConfig(1, "tiny-f32", "f32", B=2, models=(TINY,), page_size=16,
                      k_choices=(4,), ctx_lo=128, ctx_hi=128, driver_rule="alt",
                      p_argmax=0.7, alt_mode="uniform"),
    "student-bf16": WorkloadConfig(2, "student-bf16", "bf16", B=32, models=(STUDENT,), page_size=16,
                      k_choices=(8,), ctx_lo=512, ctx_hi=4096, driver_rule="T",
                      p_argmax=0.6, alt_mode="softmax", alt_temperature=1.5),
    "teacher-bf16": WorkloadConfig(3, "teacher-bf16", "bf16", B=64, models=(TEACHER,), page_size=16,
                      k_choices=(8,), ctx_lo=1024, ctx_hi=8192, driver_rule="S",
                      p_argmax=0.6, alt_mode="softmax", alt_temperature=1.5),
    "long-teacher-bf16": WorkloadConfig(4, "long-teacher-bf16", "bf16", B=16, models=(TEACHER,), page_size=16,
                      k_choices=(16,), ctx_lo=16384, ctx_hi=32768, driver_rule="S",
                      p_argmax=0.5, alt_mode="uniform", pool_tokens=2 * 1024 * 1024),
    "dual-cache-bf16": WorkloadConfig(5, "dual-cache-bf16", "bf16", B=128, models=(STUDENT, TEACHER),
                      page_size=16, k_choices=(1, 4, 8, 16), ctx_lo=256, ctx_hi=16384,
                      driver_rule="split64", p_argmax=0.6, alt_mode="softmax",
                      alt_temperature=1.5),
}

# Driver codes: 0 = the student drives (the teacher verifies),
#               1 = the teacher drives (the student verifies).
DRIVER_S = 0
DRIVER_T = 1


def scaled(cfg: WorkloadConfig, **changes) -> WorkloadConfig:
    """A copy of ``cfg`` with some fields replaced (smaller parity cases)."""
    return dataclasses.replace(cfg, **changes)


def _rng(seed: int, cfg_id: int, stream: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, cfg_id, stream]))


def _torch_gen(device: torch.device, seed: int, cfg_id: int, stream: int) -> torch.Generator:
    g = torch.Generator(device=device)
    g.manual_seed(int(np.random.SeedSequence([seed, cfg_id, stream]).generate_state(1)[0]))
    return g


def torch_dtype(name: str) -> torch.dtype:
    return {"f32": torch.float32, "bf16": torch.bfloat16}[name]


@dataclass
class ModelInputs:
    """Inputs of one verifier model's calls (attention + LM head)."""

    shape: ModelShape
    seq_ids: torch.Tensor        # int32 [n]: sequences this model verifies
    rows: torch.Tensor           # int32 [M]: batch rows of those sequences, in order
    page_table: torch.Tensor     # int32 [B, max_pages]
    num_pages: int
    k_pool: torch.Tensor         # [num_pages, Hkv, D/32, ps, 32]
    v_pool: torch.Tensor         # [num_pages, Hkv, D, ps]
    q: torch.Tensor              # [T, Hq, D] (rows of other models' sequences are zero)
    k_new: torch.Tensor          # [T, Hkv, D]
    v_new: torch.Tensor          # [T, Hkv, D]
    hidden: torch.Tensor         # [M, hidden]
    W: torch.Tensor              # [vocab, hidden]
    poison_page: int             # a pool page never assigned to a sequence


@dataclass
class Batch:
    """One verify step's batch (structure on the host, tensors on ``device``)."""

    cfg: WorkloadConfig
    ctx_lens: np.ndarray         # int32 [B]
    k: np.ndarray                # int32 [B]
    cu_q: np.ndarray             # int32 [B+1]
    driver: np.ndarray           # uint8 [B]
    verifier: np.ndarray         # int32 [B]: index into models
    seq_lens: np.ndarray         # int32 [B]: verified length before the window
    max_pages: int
    models: List[ModelInputs] = field(default_factory=list)
    u_mode: np.ndarray = None    # float64 [T]: proposal mode draw
    u_tok: np.ndarray = None     # float64 [T]: proposal token draw
    u_repl: np.ndarray = None    # float32 [B]: uniform of the replacement draw at a takeover
    eos_id: int = 0
    max_len: int = INT32_MAX

    @property
    def T(self) -> int:
        return int(self.cu_q[-1])


def _verifier_of(driver: np.ndarray, n_models: int) -> np.ndarray:
    if n_models == 1:
        return np.zeros(driver.shape, np.int32)
    # Two models = (student, teacher): the verifier is the driver's counterpart.
    return np.where(driver == DRIVER_S, 1, 0).astype(np.int32)


def make_batch(cfg: WorkloadConfig, seed: int = 0, device="cpu", poison: bool = True,
               fill_pool: bool = True) -> Batch:
    """Build one seeded batch for ``cfg`` with tensors on ``device``.

    ``poison`` fills every pool slot that holds no cached token with NaN (and
    points unused page-table entries at a NaN page), so that a read outside
    the visible keys shows up in the output.  ``fill_pool=False`` leaves the
    pool uninitialised apart from the cached tokens (used for timing runs
    whose pool is larger than what the batch reads).
    """
    device = torch.device(device)
    rng = _rng(seed, cfg.id, 0)
    B = cfg.B
    ctx = rng.integers(cfg.ctx_lo, cfg.ctx_hi + 1, size=B).astype(np.int32)
    if len(cfg.k_choices) == 1:
        k = np.full(B, cfg.k_choices[0], np.int32)
    else:
        k = rng.choice(np.asarray(cfg.k_choices, np.int32), size=B).astype(np.int32)
    cu_q = np.zeros(B + 1, np.int32)
    cu_q[1:] = np.cumsum(k)
    T = int(cu_q[-1])

    if cfg.driver_rule == "alt":
        driver = (np.arange(B) % 2).astype(np.uint8)
    elif cfg.driver_rule == "S":
        driver = np.full(B, DRIVER_S, np.uint8)
    elif cfg.driver_rule == "T":
        driver = np.full(B, DRIVER_T, np.uint8)
    elif cfg.driver_rule == "split64":
        # Bernoulli(0.5) conditioned on an exact half/half split.
        driver = np.zeros(B, np.uint8)
        driver[rng.permutation(B)[: B // 2]] = DRIVER_T
    else:
        raise ValueError(cfg.driver_rule)
    verifier = _verifier_of(driver, len(cfg.models))
    seq_lens = (ctx + 1).astype(np.int32)   # cache = verified prefix minus its last token

    ps = cfg.page_size
    max_pages = -(-(cfg.ctx_hi + max(cfg.k_choices)) // ps)
    dt = torch_dtype(cfg.dtype)
    batch = Batch(cfg, ctx, k, cu_q, driver, verifier, seq_lens, max_pages)

    for mi, shape in enumerate(cfg.models):
        mrng = _rng(seed, cfg.id, 10 + mi)
        seqs = np.nonzero(verifier == mi)[0].astype(np.int32)
        rows = np.concatenate([np.arange(cu_q[b], cu_q[b + 1]) for b in seqs]).astype(np.int32) \
            if len(seqs) else np.zeros(0, np.int32)
        need = -(-(ctx[seqs] + k[seqs]) // ps)
        total_need = int(need.sum())
        pool_pages = (cfg.pool_tokens // ps) if cfg.pool_tokens else max(2 * total_need, 8)
        num_pages = pool_pages + 1                 # the last page is never assigned
        poison_page = num_pages - 1
        perm = mrng.permutation(pool_pages)[:total_need].astype(np.int32)
        pt = np.full((B, max_pages), poison_page, np.int32)
        off = 0
        for b, n in zip(seqs, need):
            pt[b, :n] = perm[off: off + n]
            off += n

        g = _torch_gen(device, seed, cfg.id, 20 + mi)
        Hq, Hkv, D = shape.Hq, shape.Hkv, shape.D

        def randn(*size, std=1.0):
            x = torch.randn(*size, generator=g, device=device, dtype=torch.float32)
            if std != 1.0:
                x.mul_(std)
            return x.to(dt)

        fill = float("nan") if poison else 0.0
        if fill_pool:
            k_pool = torch.full((num_pages, Hkv, D // 32, ps, 32), fill, dtype=dt, device=device)
            v_pool = torch.full((num_pages, Hkv, D, ps), fill, dtype=dt, device=device)
        else:
            k_pool = torch.empty((num_pages, Hkv, D // 32, ps, 32), dtype=dt, device=device)
            v_pool = torch.empty((num_pages, Hkv, D, ps), dtype=dt, device=device)
        # Cached tokens: positions [0, L_b) of each verified sequence.
        for b in seqs:
            L = int(ctx[b])
            kc = randn(L, Hkv, D)
            vc = randn(L, Hkv, D)
            pos = torch.arange(L, device=device)
            pages = torch.from_numpy(pt[b]).to(device).long()[pos // ps]
            slots = pos % ps
            k_pool[pages, :, :, slots, :] = kc.reshape(L, Hkv, D // 32, 32)
            v_pool[pages, :, :, slots] = vc
        q = torch.zeros((T, Hq, D), dtype=dt, device=device)
        k_new = torch.zeros((T, Hkv, D), dtype=dt, device=device)
        v_new = torch.zeros((T, Hkv, D), dtype=dt, device=device)
        if len(rows):
            r = torch.from_numpy(rows).to(device).long()
            q[r] = randn(len(rows), Hq, D)
            k_new[r] = randn(len(rows), Hkv, D)
            v_new[r] = randn(len(rows), Hkv, D)
        hz = torch.randn(len(rows), shape.hidden, generator=g, device=device, dtype=torch.float32)
        hz = hz / hz.pow(2).mean(dim=1, keepdim=True).sqrt()
        hidden = hz.to(dt)
        W = randn(shape.vocab, shape.hidden, std=cfg.w_std)
        batch.models.append(ModelInputs(
            shape=shape,
            seq_ids=torch.from_numpy(seqs).to(device),
            rows=torch.from_numpy(rows).to(device),
            page_table=torch.from_numpy(pt).to(device),
            num_pages=num_pages, k_pool=k_pool, v_pool=v_pool,
            q=q, k_new=k_new, v_new=v_new, hidden=hidden, W=W,
            poison_page=poison_page))

    prng = _rng(seed, cfg.id, 1)
    batch.u_mode = prng.random(T)
    batch.u_tok = prng.random(T)
    # float32 in [0, 1): both the library and the oracle draw with this value
    batch.u_repl = np.minimum(_rng(seed, cfg.id, 2).random(cfg.B), 1.0 - 2.0 ** -24).astype(np.float32)
    batch.eos_id = cfg.models[0].vocab - 1
    return batch


def proposal_rule(cfg: WorkloadConfig):
    """The synthetic proposer's recipe: (p_argmax, alt_mode, alt_temperature)."""
    return cfg.p_argmax, cfg.alt_mode, cfg.alt_temperature


def scaled_shape(shape: ModelShape, **changes) -> ModelShape:
    """A copy of a model shape with some fields replaced (smaller parity cases)."""
    return dataclasses.replace(shape, **changes)
