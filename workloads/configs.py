"""Seeded synthetic workloads shaped like multi-turn agentic rollouts.

The paper measures on WebShop, AlfWorld, OSWorld and ScienceBoard trajectories
(Section 6.1; per-workload turn and token counts in the task-statistics table of
Appendix C).  Those datasets are not available here, and the attention path only
needs their shapes, so every workload below is synthetic: lengths drawn from the
stated laws, Q/K/V ~ N(0,1) rounded to bf16, and physical pages scattered over a
shared pool.  The workloads are:

  tiny_extend        4 tasks, 8 q / 2 kv heads, d=64; fixed prefix/extend lengths
  agent_resume_7b    64 tasks, 28 q / 4 kv heads (7B-class layer), d=128; prefix
                     U{2048..16384}, extend (observation) log-uniform 64..2048
  resumed_decode     256 tasks, 32 q / 8 kv heads, d=128; context lognormal
                     (median 6144, sigma 0.7) clipped to [1024, 32768]; one token each
  multimodal_resume  32 tasks, 32 q / 8 kv heads, d=128; prefix U{4096..24576},
                     extend U{1024..4096}; K rows x4 on 10% of positions
  long_horizon       32 tasks, 64 q / 8 kv heads, d=128; prefix U{32768..98304},
                     extend U{256..1024}; pool 90% occupied; then 8 decode steps
  grpo_group_decode  32 GRPO groups x 8 trajectories, 32 q / 8 kv heads, d=128; each
                     group's prompt (U{2048..6144}, page-aligned) sits in pages all its
                     trajectories share; each trajectory's own context after it is
                     lognormal (median 3072, sigma 0.7) clipped to [256, 16384]; one
                     decoded token each
  multimodal_prune_resume
                     32 tasks, 32 q / 8 kv heads, d=128; prompt U{512..2048}, then ten
                     turns of (1196-token screenshot, U{64..256} text tokens); the tenth
                     image prunes the five oldest screenshots, so everything after the
                     prompt moves: the resume is an extend with P = prompt and E = the
                     five old turns' text + the five kept turns, written over pages
                     that still hold the pre-prune context

This module only draws inputs (lengths, page placement, tensor values); it holds
none of the attention arithmetic.
"""
from __future__ import annotations

import dataclasses
import hashlib
import math
from dataclasses import dataclass, field

import numpy as np

from . import _native

# Stream ids of the counter-based generator (stream_a); stream_b is the task index.
TENSOR_Q = 1
TENSOR_K = 2
TENSOR_V = 3

KILO = 1024  # "2k", "16k", "96k" ... are read as multiples of 1024


@dataclass(frozen=True)
class Spec:
    key: str
    index: int
    text: str
    num_tasks: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    page_size: int
    kind: str  # "extend" | "decode" | "long_horizon"
    prefix: tuple = ()  # ("fixed", values) | ("uniform", lo, hi)
    extend: tuple = ()  # ("fixed", values) | ("uniform", lo, hi) | ("loguniform", lo, hi)
    context: tuple = ()  # decode only: ("lognormal", median, sigma, lo, hi)
    pool: tuple = ("fragmented", 1.1)  # ("perm", N) | ("fragmented", f) | ("occupied", f)
    outlier_frac: float = 0.0
    outlier_scale: float = 1.0
    decode_steps: int = 0
    prune: tuple = ()    # prune_resume: (images, keep, image_tokens, ("uniform", lo, hi) text)
    group_size: int = 0  # > 0: consecutive tasks form GRPO groups sharing a prompt prefix
    shared: tuple = ()   # group_decode: ("uniform", lo, hi) prompt length, rounded to pages
    salt: int = 0  # 0 for the full-size workload; shrunken variants use their own seeds

    @property
    def group(self) -> int:
        return self.num_q_heads // self.num_kv_heads

    def shrunk(self, num_tasks: int, length_div: int, salt: int = 1) -> "Spec":
        """A smaller workload with the same structure, for CPU-sized oracle checks."""

        def div_range(law):
            if not law:
                return law
            if law[0] == "fixed":
                return ("fixed", tuple(max(1, v // length_div) for v in law[1][:num_tasks]))
            if law[0] in ("uniform", "loguniform"):
                return (law[0], max(1, law[1] // length_div), max(1, law[2] // length_div))
            if law[0] == "lognormal":
                return ("lognormal", max(2, law[1] // length_div), law[2],
                        max(2, law[3] // length_div), max(2, law[4] // length_div))
            raise ValueError(law)

        pool = self.pool
        if pool[0] == "perm":
            pool = ("fragmented", 1.5)
        prune = self.prune
        if prune:
            prune = (prune[0], prune[1], max(1, prune[2] // length_div), div_range(prune[3]))
        return dataclasses.replace(
            self, num_tasks=num_tasks, prefix=div_range(self.prefix),
            extend=div_range(self.extend), context=div_range(self.context), pool=pool,
            shared=div_range(self.shared), prune=prune, salt=salt)


SPECS = {
    "tiny_extend": Spec(
        key="tiny_extend", index=1,
        text=("Tiny extend-attention: 4 tasks, 8 query heads / 2 KV heads (GQA), head_dim 64, "
              "page size 16, prefix lens {37,100,250,511}, extend lens {5,17,64,128}, causal; "
              "Q/K/V bf16 ~ N(0,1), softmax scale 1/sqrt(64); physical pages a seeded random "
              "permutation of a 128-page pool"),
        num_tasks=4, num_q_heads=8, num_kv_heads=2, head_dim=64, page_size=16, kind="extend",
        prefix=("fixed", (37, 100, 250, 511)), extend=("fixed", (5, 17, 64, 128)),
        pool=("perm", 128)),
    "agent_resume_7b": Spec(
        key="agent_resume_7b", index=2,
        text=("Agent resume, 7B-class layer: 64 tasks, 28 query / 4 KV heads, head_dim 128, "
              "page 16, prefix lens uniform 2k-16k, extend (observation) lens log-uniform "
              "64-2048, bf16 ~ N(0,1), causal, fragmented random page placement; also full "
              "re-prefill of the same sequences for comparison"),
        num_tasks=64, num_q_heads=28, num_kv_heads=4, head_dim=128, page_size=16, kind="extend",
        prefix=("uniform", 2 * KILO, 16 * KILO), extend=("loguniform", 64, 2048),
        pool=("fragmented", 1.1)),
    "resumed_decode": Spec(
        key="resumed_decode", index=3,
        text=("Resumed decode: 256 concurrent tasks, 1 query token each, 32 query / 8 KV heads, "
              "head_dim 128, page 16, context lens lognormal (median 6k, clipped 1k-32k), "
              "bf16 ~ N(0,1), split-K over context"),
        num_tasks=256, num_q_heads=32, num_kv_heads=8, head_dim=128, page_size=16, kind="decode",
        context=("lognormal", 6 * KILO, 0.7, 1 * KILO, 32 * KILO), pool=("fragmented", 1.1)),
    "multimodal_resume": Spec(
        key="multimodal_resume", index=4,
        text=("Multi-modal observation resume: 32 tasks, 32 query / 8 KV heads, head_dim 128, "
              "page 16, prefix lens uniform 4k-24k, extend lens uniform 1024-4096 "
              "(image-patch-sized chunks), bf16 with K rows scaled x4 on 10% of positions "
              "(outlier tokens), causal"),
        num_tasks=32, num_q_heads=32, num_kv_heads=8, head_dim=128, page_size=16, kind="extend",
        prefix=("uniform", 4 * KILO, 24 * KILO), extend=("uniform", 1024, 4096),
        pool=("fragmented", 1.1), outlier_frac=0.1, outlier_scale=4.0),
    "long_horizon": Spec(
        key="long_horizon", index=5,
        text=("Long-horizon agent: 32 tasks, 64 query / 8 KV heads, head_dim 128, page 16, "
              "prefix lens uniform 32k-96k, extend lens uniform 256-1024, bf16 ~ N(0,1); "
              "KV-append of extend tokens into a 90%-occupied shuffled page pool, followed by "
              "extend-attention and then 8 decode steps per task"),
        num_tasks=32, num_q_heads=64, num_kv_heads=8, head_dim=128, page_size=16,
        kind="long_horizon", prefix=("uniform", 32 * KILO, 96 * KILO), extend=("uniform", 256, 1024),
        pool=("occupied", 0.9), decode_steps=8),
    "grpo_group_decode": Spec(
        key="grpo_group_decode", index=6,
        text=("GRPO group decode (shared-prompt attention): 32 groups of 8 trajectories, "
              "32 query / 8 KV heads, head_dim 128, page 16; each group's prompt, uniform "
              "2k-6k tokens rounded down to whole pages, is stored once in pages every "
              "trajectory of the group maps; each trajectory's own context after it is "
              "lognormal (median 3k, sigma 0.7) clipped to [256, 16k]; one decoded token "
              "per trajectory; bf16 ~ N(0,1)"),
        num_tasks=256, num_q_heads=32, num_kv_heads=8, head_dim=128, page_size=16,
        kind="group_decode", context=("lognormal", 3 * KILO, 0.7, 256, 16 * KILO),
        group_size=8, shared=("uniform", 2 * KILO, 6 * KILO), pool=("fragmented", 1.1)),
    "multimodal_prune_resume": Spec(
        key="multimodal_prune_resume", index=7,
        text=("Multi-modal sliding-window prune resume: 32 tasks, 32 query / 8 KV heads, "
              "head_dim 128, page 16; prompt uniform 512-2048 tokens, then ten turns of one "
              "1280x720 screenshot (1196 tokens at 28-pixel patches) and uniform 64-256 text "
              "tokens; on the tenth image the five oldest screenshots are pruned, and the "
              "resume re-encodes everything after the prompt (the old turns' text and the "
              "five kept turns) over the pages that held the pre-prune context; also full "
              "re-prefill of the pruned sequence; bf16 ~ N(0,1)"),
        num_tasks=32, num_q_heads=32, num_kv_heads=8, head_dim=128, page_size=16,
        kind="prune_resume", prefix=("uniform", 512, 2048),
        prune=(10, 5, 1196, ("uniform", 64, 256)), pool=("fragmented", 1.1)),
}


def _ceil_div(a, b):
    return -(-a // b)


@dataclass
class Workload:
    """Drawn lengths, page placement and lazily generated tensors of one workload.

    Positions of task b: 0 .. prefix_lens[b]-1 are the retained prefix,
    prefix_lens[b] .. prefix_lens[b]+extend_lens[b]-1 the resumed (appended) tokens, and
    for long_horizon the next decode_steps positions are the decoded tokens.
    """

    spec: Spec
    prefix_lens: np.ndarray
    extend_lens: np.ndarray
    block_table: np.ndarray
    num_pages: int
    seeds: dict
    outliers: list = field(default_factory=list)
    group_start: np.ndarray | None = None  # GRPO groups: tasks group_start[g] .. [g+1]-1
    shared_lens: np.ndarray | None = None  # positions 0 .. shared-1 in the group's pages
    stale_lens: np.ndarray | None = None   # prune resume: context length before the prune

    # ---- shape helpers -------------------------------------------------------------
    @property
    def num_tasks(self):
        return self.spec.num_tasks

    @property
    def seq_lens(self) -> np.ndarray:
        return (self.prefix_lens + self.extend_lens).astype(np.int32)

    @property
    def final_lens(self) -> np.ndarray:
        """Longest context the task's pages hold at any point (they are mapped up to it)."""
        n = self.seq_lens.astype(np.int64) + self.spec.decode_steps
        if self.stale_lens is not None:
            n = np.maximum(n, self.stale_lens)
        return n.astype(np.int32)

    @property
    def sm_scale(self) -> float:
        return 1.0 / math.sqrt(self.spec.head_dim)

    @property
    def bt_stride(self) -> int:
        return int(self.block_table.shape[1])

    def lens_digest(self) -> str:
        h = hashlib.sha256()
        h.update(self.prefix_lens.astype("<i4").tobytes())
        h.update(self.extend_lens.astype("<i4").tobytes())
        return h.hexdigest()[:16]

    # ---- tensor slices (bf16 bit patterns as uint16) --------------------------------
    def group_of(self, b: int) -> int:
        return int(np.searchsorted(self.group_start, b, side="right") - 1)

    def _rows(self, tensor: int, heads: int, b: int, t0: int, t1: int, out=None) -> np.ndarray:
        d = self.spec.head_dim
        rows = max(0, t1 - t0)
        if out is None:
            out = np.empty((rows, heads, d), dtype=np.uint16)
        flat = out.reshape(-1)
        # K/V of a shared prompt prefix come from the group's own stream (ids after the
        # tasks'), so every trajectory of the group holds the same values there
        sh = 0
        if self.shared_lens is not None and tensor != TENSOR_Q:
            sh = int(self.shared_lens[self.group_of(b)])
        cut = min(max(t0, sh), t1)
        if cut > t0:
            g = self.num_tasks + self.group_of(b)
            _native.normal_bf16(self.seeds[tensor], tensor, g, t0 * heads * d,
                                (cut - t0) * heads * d, out=flat[:(cut - t0) * heads * d])
        if t1 > cut:
            _native.normal_bf16(self.seeds[tensor], tensor, b, cut * heads * d,
                                (t1 - cut) * heads * d, out=flat[(cut - t0) * heads * d:])
        return flat.reshape(rows, heads, d)

    def stale_rows(self, which: str, b: int, t0: int, t1: int) -> np.ndarray:
        """K or V the pool held at positions t0..t1-1 before a prune (the pruned and the
        old, differently encoded turns); drawn from streams of their own."""
        tensor = {"k": TENSOR_K, "v": TENSOR_V}[which]
        d, heads = self.spec.head_dim, self.spec.num_kv_heads
        rows = max(0, t1 - t0)
        flat = _native.normal_bf16(self.seeds[tensor], tensor, 2 * self.num_tasks + b,
                                   t0 * heads * d, rows * heads * d)
        return flat.reshape(rows, heads, d)

    def stale_ranges(self):
        """Positions that held pre-prune K/V when the resume starts: prompt end .. old end."""
        return [(int(p), int(s)) for p, s in zip(self.prefix_lens, self.stale_lens)]

    def stale_packed(self, which: str) -> np.ndarray:
        parts = [self.stale_rows(which, b, t0, t1) for b, (t0, t1) in enumerate(self.stale_ranges())]
        if not parts:
            return np.zeros((0, self.spec.num_kv_heads, self.spec.head_dim), np.uint16)
        return np.concatenate(parts)

    def q_rows(self, b: int, t0: int, t1: int, out=None) -> np.ndarray:
        return self._rows(TENSOR_Q, self.spec.num_q_heads, b, t0, t1, out)

    def k_rows(self, b: int, t0: int, t1: int, out=None) -> np.ndarray:
        k = self._rows(TENSOR_K, self.spec.num_kv_heads, b, t0, t1, out)
        if self.outliers:
            sel = self.outliers[b][t0:t1]
            if sel.any():
                f = _bf16_to_f32(k[sel]) * np.float32(self.spec.outlier_scale)
                k[sel] = _f32_to_bf16_exact(f)
        return k

    def v_rows(self, b: int, t0: int, t1: int, out=None) -> np.ndarray:
        return self._rows(TENSOR_V, self.spec.num_kv_heads, b, t0, t1, out)

    def packed(self, which: str, ranges) -> np.ndarray:
        """Concatenate per-task row ranges [(t0, t1)] of 'q', 'k' or 'v' in task order."""
        fn = {"q": self.q_rows, "k": self.k_rows, "v": self.v_rows}[which]
        heads = self.spec.num_q_heads if which == "q" else self.spec.num_kv_heads
        total = sum(max(0, t1 - t0) for t0, t1 in ranges)
        out = np.empty((total, heads, self.spec.head_dim), dtype=np.uint16)
        row = 0
        for b, (t0, t1) in enumerate(ranges):
            n = max(0, t1 - t0)
            if n:
                fn(b, t0, t1, out=out[row:row + n])
            row += n
        return out

    def prefix_ranges(self):
        return [(0, int(p)) for p in self.prefix_lens]

    def extend_ranges(self):
        return [(int(p), int(p + e)) for p, e in zip(self.prefix_lens, self.extend_lens)]

    def full_ranges(self):
        return [(0, int(l)) for l in self.seq_lens]

    def decode_ranges(self, step: int):
        return [(int(l) + step, int(l) + step + 1) for l in self.seq_lens]

    def remap_pages(self, perm: np.ndarray) -> "Workload":
        """The same workload with physical page i moved to page perm[i]."""
        bt = self.block_table.copy()
        live = bt >= 0
        bt[live] = perm[bt[live]]
        return dataclasses.replace(self, block_table=bt)


def _bf16_to_f32(a: np.ndarray) -> np.ndarray:
    return (a.astype(np.uint32) << 16).view(np.float32)


def _f32_to_bf16_exact(f: np.ndarray) -> np.ndarray:
    u = f.astype(np.float32).view(np.uint32)
    assert not (u & 0xFFFF).any(), "scaled value is not exactly representable in bf16"
    return (u >> 16).astype(np.uint16)


def _draw_group_lengths(spec: Spec, rng: np.random.Generator):
    """GRPO groups: per-group prompt lengths (whole pages), per-trajectory own context."""
    b, gsz, ps = spec.num_tasks, spec.group_size, spec.page_size
    assert b % gsz == 0
    ng = b // gsz
    _, lo, hi = spec.shared
    shared = rng.integers(lo, hi, size=ng, endpoint=True) // ps * ps
    _, median, sigma, clo, chi = spec.context
    own = np.clip(np.rint(rng.lognormal(math.log(median), sigma, size=b)), clo, chi)
    ctx = np.repeat(shared, gsz).astype(np.int64) + own.astype(np.int64)
    group_start = np.arange(0, b + 1, gsz, dtype=np.int32)
    # the newest token of each trajectory is the one being decoded: it is appended first
    return (ctx - 1).astype(np.int32), np.ones(b, dtype=np.int32), group_start, shared.astype(np.int32)


def _prune_lengths(prompt, texts, images: int, keep: int, image_tokens: int):
    """Prompt, then turns of (screenshot, text).  With `images` screenshots in context the
    oldest images - keep are dropped; their turns' text stays.  Returns (P, E, old length):
    P = position of the first dropped token, E = tokens after it in the pruned sequence."""
    prompt = np.asarray(prompt, dtype=np.int64)
    texts = np.asarray(texts, dtype=np.int64).reshape(prompt.size, images)
    old_len = prompt + images * image_tokens + texts.sum(axis=1)
    if keep >= images:
        return prompt.astype(np.int32), np.zeros_like(prompt, np.int32), old_len.astype(np.int32)
    tail = old_len - prompt - (images - keep) * image_tokens
    return prompt.astype(np.int32), tail.astype(np.int32), old_len.astype(np.int32)


def _draw_prune_lengths(spec: Spec, rng: np.random.Generator):
    b = spec.num_tasks
    images, keep, img_tok, text = spec.prune
    prompt = rng.integers(spec.prefix[1], spec.prefix[2], size=b, endpoint=True)
    texts = rng.integers(text[1], text[2], size=(b, images), endpoint=True)
    return _prune_lengths(prompt, texts, images, keep, img_tok)


def _draw_lengths(spec: Spec, rng: np.random.Generator):
    b = spec.num_tasks
    if spec.kind == "decode":
        law = spec.context
        assert law[0] == "lognormal"
        _, median, sigma, lo, hi = law
        ctx = np.rint(rng.lognormal(math.log(median), sigma, size=b))
        ctx = np.clip(ctx, lo, hi).astype(np.int64)
        # the newest token of each task is the one being decoded: it is appended first
        return (ctx - 1).astype(np.int32), np.ones(b, dtype=np.int32)

    def draw(law):
        if law[0] == "fixed":
            vals = np.asarray(law[1][:b], dtype=np.int64)
            assert vals.size == b
            return vals
        if law[0] == "uniform":
            return rng.integers(law[1], law[2], size=b, endpoint=True)
        if law[0] == "loguniform":
            lo, hi = law[1], law[2]
            v = np.floor(np.exp(rng.uniform(math.log(lo), math.log(hi), size=b)))
            return np.clip(v, lo, hi).astype(np.int64)
        raise ValueError(law)

    p = draw(spec.prefix)
    e = draw(spec.extend)
    return p.astype(np.int32), e.astype(np.int32)


def _place_group_pages(spec: Spec, prefix, extend, group_start, shared, rng):
    """Fragmented pool; a group's prompt pages are allocated once and mapped by all of its
    trajectories, then each trajectory gets its own pages."""
    ps = spec.page_size
    final = prefix.astype(np.int64) + extend
    need = [_ceil_div(int(f), ps) for f in final]
    stride = max(need)
    bt = np.full((spec.num_tasks, stride), -1, dtype=np.int32)
    ng = len(shared)
    total = sum(int(s) // ps for s in shared) + sum(
        need[b] - int(shared[g]) // ps for g in range(ng)
        for b in range(group_start[g], group_start[g + 1]))
    n = int(math.ceil(spec.pool[1] * total))
    perm = rng.permutation(n).astype(np.int32)
    at = 0
    for g in range(ng):
        sp = int(shared[g]) // ps
        pages = perm[at:at + sp]
        at += sp
        for b in range(group_start[g], group_start[g + 1]):
            bt[b, :sp] = pages
            k = need[b] - sp
            bt[b, sp:sp + k] = perm[at:at + k]
            at += k
    return bt, n


def _place_pages(spec: Spec, prefix, extend, rng: np.random.Generator, final=None):
    ps = spec.page_size
    if final is None:
        final = prefix.astype(np.int64) + extend + spec.decode_steps
    need = [_ceil_div(int(f), ps) for f in final]
    stride = max(1, max(need) if need else 1)
    bt = np.full((spec.num_tasks, stride), -1, dtype=np.int32)
    kind = spec.pool[0]
    if kind in ("perm", "fragmented"):
        total = int(sum(need))
        n = spec.pool[1] if kind == "perm" else int(math.ceil(spec.pool[1] * total))
        assert n >= total, "pool too small"
        perm = rng.permutation(n).astype(np.int32)
        at = 0
        for b, k in enumerate(need):
            bt[b, :k] = perm[at:at + k]
            at += k
        return bt, n
    if kind == "occupied":
        pref_pages = [_ceil_div(int(p), ps) for p in prefix]
        n_pref = int(sum(pref_pages))
        n = int(math.ceil(n_pref / spec.pool[1]))
        perm = rng.permutation(n).astype(np.int32)
        at = 0
        for b, k in enumerate(pref_pages):
            bt[b, :k] = perm[at:at + k]
            at += k
        free = list(perm[at:])
        free.reverse()  # pop() takes from the front of the shuffled free list
        # the appended tokens first fill each task's partial last page, then take free pages
        for b in range(spec.num_tasks):
            for lp in range(pref_pages[b], _ceil_div(int(prefix[b] + extend[b]), ps)):
                bt[b, lp] = free.pop()
        # decode steps, one token per task per step, in task order
        for s in range(spec.decode_steps):
            for b in range(spec.num_tasks):
                pos = int(prefix[b] + extend[b]) + s
                if pos % ps == 0:
                    bt[b, pos // ps] = free.pop()
        return bt, n
    raise ValueError(spec.pool)


def make_workload(spec: Spec | str) -> Workload:
    """Draw one workload.  Same spec => same lengths, pages and tensor values."""
    if isinstance(spec, str):
        spec = SPECS[spec]
    ss = np.random.SeedSequence([2608, 10402, spec.index, spec.salt])
    c_lens, c_pages, c_q, c_k, c_v, c_out = ss.spawn(6)
    group_start = shared = stale = None
    if spec.kind == "prune_resume":
        prefix, extend, stale = _draw_prune_lengths(spec, np.random.Generator(np.random.PCG64(c_lens)))
        # the task's pages cover its context before the prune; the resumed sequence reuses
        # the first of them
        bt, n_pages = _place_pages(spec, prefix, extend,
                                   np.random.Generator(np.random.PCG64(c_pages)),
                                   final=stale.astype(np.int64))
    elif spec.kind == "group_decode":
        prefix, extend, group_start, shared = _draw_group_lengths(
            spec, np.random.Generator(np.random.PCG64(c_lens)))
        bt, n_pages = _place_group_pages(spec, prefix, extend, group_start, shared,
                                         np.random.Generator(np.random.PCG64(c_pages)))
    else:
        prefix, extend = _draw_lengths(spec, np.random.Generator(np.random.PCG64(c_lens)))
        bt, n_pages = _place_pages(spec, prefix, extend,
                                   np.random.Generator(np.random.PCG64(c_pages)))

    def seed64(c):
        w = c.generate_state(2, np.uint32)
        return int(w[0]) | (int(w[1]) << 32)

    seeds = {TENSOR_Q: seed64(c_q), TENSOR_K: seed64(c_k), TENSOR_V: seed64(c_v)}
    outliers = []
    if spec.outlier_frac > 0:
        rng = np.random.Generator(np.random.PCG64(c_out))
        final = prefix.astype(np.int64) + extend + spec.decode_steps
        outliers = [rng.random(int(f)) < spec.outlier_frac for f in final]
    return Workload(spec=spec, prefix_lens=prefix, extend_lens=extend, block_table=bt,
                    num_pages=int(n_pages), seeds=seeds, outliers=outliers,
                    group_start=group_start, shared_lens=shared, stale_lens=stale)


def custom_workload(num_q_heads: int, num_kv_heads: int, head_dim: int, prefix_lens,
                    extend_lens, num_pages: int | None = None, seed: int = 0,
                    decode_steps: int = 0, outlier_frac: float = 0.0) -> Workload:
    """A workload with explicit lengths (edge cases: empty extends, fresh tasks, ...)."""
    prefix = np.asarray(prefix_lens, dtype=np.int32)
    extend = np.asarray(extend_lens, dtype=np.int32)
    spec = Spec(key="custom", index=100 + seed, text="explicit lengths", num_tasks=int(prefix.size),
                num_q_heads=num_q_heads, num_kv_heads=num_kv_heads, head_dim=head_dim,
                page_size=16, kind="extend", prefix=("fixed", tuple(int(x) for x in prefix)),
                extend=("fixed", tuple(int(x) for x in extend)),
                pool=("fragmented", 1.25) if num_pages is None else ("perm", num_pages),
                decode_steps=decode_steps, outlier_frac=outlier_frac,
                outlier_scale=4.0 if outlier_frac else 1.0, salt=seed)
    if num_pages is not None:
        need = sum(_ceil_div(int(p + e + decode_steps), 16) for p, e in zip(prefix, extend))
        if need > num_pages:
            spec = dataclasses.replace(spec, pool=("fragmented", 1.25))
    return make_workload(spec)


def custom_group_workload(num_q_heads: int, num_kv_heads: int, head_dim: int, group_sizes,
                          shared_lens, own_lens, seed: int = 0) -> Workload:
    """GRPO groups with explicit sizes, shared prompt lengths (page multiples) and each
    trajectory's own context length after the prompt (>= 1: the decoded token)."""
    sizes = [int(x) for x in group_sizes]
    shared = np.asarray(shared_lens, dtype=np.int32)
    own = np.asarray(own_lens, dtype=np.int64)
    assert len(shared) == len(sizes) and own.size == sum(sizes) and (own >= 1).all()
    assert (shared % 16 == 0).all()
    group_start = np.concatenate([[0], np.cumsum(sizes)]).astype(np.int32)
    ctx = np.repeat(shared, sizes).astype(np.int64) + own
    spec = Spec(key="custom_group", index=200 + seed, text="explicit GRPO groups",
                num_tasks=int(own.size), num_q_heads=num_q_heads, num_kv_heads=num_kv_heads,
                head_dim=head_dim, page_size=16, kind="group_decode",
                group_size=max(sizes), pool=("fragmented", 1.25), salt=seed)
    ss = np.random.SeedSequence([2608, 10402, spec.index, spec.salt])
    c_lens, c_pages, c_q, c_k, c_v, c_out = ss.spawn(6)
    prefix = (ctx - 1).astype(np.int32)
    extend = np.ones(own.size, dtype=np.int32)
    bt, n_pages = _place_group_pages(spec, prefix, extend, group_start, shared,
                                     np.random.Generator(np.random.PCG64(c_pages)))

    def seed64(c):
        w = c.generate_state(2, np.uint32)
        return int(w[0]) | (int(w[1]) << 32)

    seeds = {TENSOR_Q: seed64(c_q), TENSOR_K: seed64(c_k), TENSOR_V: seed64(c_v)}
    return Workload(spec=spec, prefix_lens=prefix, extend_lens=extend, block_table=bt,
                    num_pages=int(n_pages), seeds=seeds, group_start=group_start,
                    shared_lens=shared)


def custom_prune_workload(num_q_heads: int, num_kv_heads: int, head_dim: int, prompt_lens,
                          texts, images: int = 10, keep: int = 5, image_tokens: int = 1196,
                          seed: int = 0) -> Workload:
    """Sliding-window prune resume with explicit prompt lengths and per-turn text lengths
    (texts[b][i] = text tokens of turn i of task b, `images` turns per task)."""
    prompt = np.asarray(prompt_lens, dtype=np.int64)
    prefix, extend, stale = _prune_lengths(prompt, texts, images, keep, image_tokens)
    spec = Spec(key="custom_prune", index=300 + seed, text="explicit prune resume",
                num_tasks=int(prompt.size), num_q_heads=num_q_heads, num_kv_heads=num_kv_heads,
                head_dim=head_dim, page_size=16, kind="prune_resume",
                prune=(images, keep, image_tokens, ("fixed", ())), pool=("fragmented", 1.25),
                salt=seed)
    ss = np.random.SeedSequence([2608, 10402, spec.index, spec.salt])
    c_lens, c_pages, c_q, c_k, c_v, c_out = ss.spawn(6)
    bt, n_pages = _place_pages(spec, prefix, extend, np.random.Generator(np.random.PCG64(c_pages)),
                               final=stale.astype(np.int64))

    def seed64(c):
        w = c.generate_state(2, np.uint32)
        return int(w[0]) | (int(w[1]) << 32)

    seeds = {TENSOR_Q: seed64(c_q), TENSOR_K: seed64(c_k), TENSOR_V: seed64(c_v)}
    return Workload(spec=spec, prefix_lens=prefix, extend_lens=extend, block_table=bt,
                    num_pages=int(n_pages), seeds=seeds, stale_lens=stale)
