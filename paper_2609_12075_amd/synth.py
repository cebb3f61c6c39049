"""Model shapes and seeded synthetic inputs for the VLA serving hot path.

This module holds no arithmetic of the method. It defines

* the model configurations (shapes of the two-stage VLA: a VLM that encodes
  the camera frames and the instruction text into per-layer prefix state, and an action
  diffusion transformer that runs a few denoising steps, paper Section 2.1),
* the canonical order and shapes of the parameter tensors, and
* seeded generators for parameters and request inputs.

Both the CPU oracle and the GPU library consume what this module produces;
neither side's arithmetic lives here. Random values are drawn with numpy's
PCG64 from ``SeedSequence(base, spawn_key=(i,))`` so that tensor ``i`` (or
batch row ``i``) is the same whatever else is drawn.

Parameter storage: every matrix is stored ``[in, out]`` row-major in fp32,
tensors concatenated in the order ``weight_schema`` lists them. Matrices,
biases, embeddings, position tables and modulation weights are N(0, 0.02);
norm gains are 1 + N(0, 0.02).
"""
from __future__ import annotations

import dataclasses
from typing import Dict, List, Tuple

import numpy as np

DTYPE_F32 = 0
DTYPE_BF16 = 1
HEAD_JOINT = 0   # action expert attends over [prefix KV ; action tokens]
HEAD_DIT = 1     # DiT action head: adaLN self-attention + cross-attention


@dataclasses.dataclass(frozen=True)
class VLAConfig:
    name: str
    dtype: int
    n_img: int
    img_hw: int
    patch: int
    vit_layers: int
    vit_d: int
    vit_heads: int
    vit_mlp: int
    n_text: int
    vocab: int
    llm_layers: int
    llm_d: int
    n_q: int
    n_kv: int
    head_dim: int
    llm_mlp: int
    head_kind: int
    act_layers: int
    act_d: int
    act_heads: int
    act_mlp: int
    horizon: int
    action_dim: int
    state_dim: int
    max_batch: int
    steps: int
    seed: int
    rope_base: float = 10000.0
    norm_eps: float = 1e-6
    time_dim: int = 0          # sinusoid width for the DiT time MLP (0: act_d)
    pix_shuffle: int = 1       # s x s blocks of encoder tokens merged into one image token (1: none)

    # ---- derived sizes (pure bookkeeping) ----
    @property
    def patch_grid(self) -> int:
        return self.img_hw // self.patch

    @property
    def patch_tokens(self) -> int:
        """Patch tokens per image (the vision encoder's sequence)."""
        return self.patch_grid ** 2

    @property
    def tokens_per_img(self) -> int:
        """Image tokens per image in the LLM prefix."""
        return self.patch_tokens // (self.pix_shuffle ** 2)

    @property
    def n_img_tokens(self) -> int:
        return self.n_img * self.tokens_per_img

    @property
    def prefix_len(self) -> int:
        return self.n_img_tokens + self.n_text

    @property
    def patch_dim(self) -> int:
        return 3 * self.patch * self.patch

    @property
    def embed_d(self) -> int:
        """Width of the patch embedding (the ViT width, or the LLM width when
        there is no vision encoder)."""
        return self.vit_d if self.vit_layers > 0 else self.llm_d

    @property
    def n_tokens_act(self) -> int:
        """Tokens the action stage processes per request."""
        return self.horizon + (1 if self.head_kind == HEAD_DIT else 0)

    @property
    def tdim(self) -> int:
        return self.time_dim if self.time_dim else self.act_d

    def with_(self, **kw) -> "VLAConfig":
        return dataclasses.replace(self, **kw)


CONFIGS: Dict[str, VLAConfig] = {}

# Tiny fp32 VLA (batch 1 in its workload; max_batch 4 lets tests batch it).
CONFIGS["tiny"] = VLAConfig(
    name="tiny", dtype=DTYPE_F32, n_img=1, img_hw=64, patch=8,
    vit_layers=0, vit_d=0, vit_heads=0, vit_mlp=0,
    n_text=16, vocab=1000, llm_layers=2, llm_d=256, n_q=4, n_kv=4, head_dim=64,
    llm_mlp=1024, head_kind=HEAD_JOINT, act_layers=2, act_d=128, act_heads=4,
    act_mlp=512, horizon=8, action_dim=7, state_dim=0, max_batch=4, steps=4,
    seed=0)

# SmolVLA-shaped, bf16, batch 1-16.
CONFIGS["smolvla"] = VLAConfig(
    name="smolvla", dtype=DTYPE_BF16, n_img=3, img_hw=64, patch=8,
    vit_layers=0, vit_d=0, vit_heads=0, vit_mlp=0,
    n_text=48, vocab=1000, llm_layers=16, llm_d=960, n_q=15, n_kv=5, head_dim=64,
    llm_mlp=2560, head_kind=HEAD_JOINT, act_layers=16, act_d=720, act_heads=15,
    act_mlp=1920, horizon=50, action_dim=32, state_dim=0, max_batch=16, steps=10,
    seed=1)

# SmolVLA-shaped with its whole vision encoder (a SigLIP-like ViT on 512 x 512
# images, patch 16, whose 32 x 32 patch tokens are merged in 4 x 4 blocks into
# 64 image tokens before the projection to the LLM width): the prefix keeps
# 3 x 64 image tokens + 48 text tokens, as in the configuration above.
CONFIGS["smolvla_vit"] = CONFIGS["smolvla"].with_(
    name="smolvla_vit", img_hw=512, patch=16, vit_layers=12, vit_d=768, vit_heads=12, vit_mlp=3072,
    pix_shuffle=4, seed=4)

# pi0-shaped, bf16, batch 1-32.
CONFIGS["pi0"] = VLAConfig(
    name="pi0", dtype=DTYPE_BF16, n_img=3, img_hw=224, patch=14,
    vit_layers=27, vit_d=1152, vit_heads=16, vit_mlp=4304,
    n_text=48, vocab=1000, llm_layers=18, llm_d=2048, n_q=8, n_kv=1, head_dim=256,
    llm_mlp=16384, head_kind=HEAD_JOINT, act_layers=18, act_d=1024, act_heads=8,
    act_mlp=4096, horizon=50, action_dim=32, state_dim=0, max_batch=32, steps=10,
    seed=2)

# GR00T-like DiT action head, bf16, batch 1-32.
CONFIGS["gr00t"] = VLAConfig(
    name="gr00t", dtype=DTYPE_BF16, n_img=1, img_hw=224, patch=14,
    vit_layers=27, vit_d=1152, vit_heads=16, vit_mlp=4304,
    n_text=40, vocab=1000, llm_layers=12, llm_d=2048, n_q=8, n_kv=1, head_dim=256,
    llm_mlp=16384, head_kind=HEAD_DIT, act_layers=16, act_d=1024, act_heads=32,
    act_mlp=4096, horizon=16, action_dim=32, state_dim=32, max_batch=32, steps=4,
    seed=3, time_dim=256)


def reduced(cfg: VLAConfig, vit_layers=None, llm_layers=2, act_layers=2,
            max_batch=None) -> VLAConfig:
    """Same widths, fewer layers: a variant the fp64 oracle finishes in seconds."""
    vl = cfg.vit_layers if vit_layers is None else vit_layers
    if cfg.vit_layers > 0:
        vl = max(1, vl)
    return cfg.with_(name=cfg.name + "-reduced", vit_layers=vl,
                     llm_layers=llm_layers, act_layers=act_layers,
                     max_batch=cfg.max_batch if max_batch is None else max_batch,
                     seed=cfg.seed + 100)


# ---------------------------------------------------------------------------
# Parameter schema
# ---------------------------------------------------------------------------
MAT, VEC, GAIN = "mat", "vec", "gain"


def weight_schema(c: VLAConfig) -> List[Tuple[str, Tuple[int, ...], str]]:
    """Canonical (name, shape, kind) list. The flat parameter buffer is these
    tensors concatenated in this order, each row-major fp32."""
    s: List[Tuple[str, Tuple[int, ...], str]] = []
    add = lambda n, sh, k: s.append((n, tuple(int(x) for x in sh), k))
    E, T = c.embed_d, c.patch_tokens
    # vision front-end
    add("patch.w", (c.patch_dim, E), MAT)
    add("patch.b", (E,), VEC)
    add("patch.pos", (T, E), VEC)
    for l in range(c.vit_layers):
        d, f = c.vit_d, c.vit_mlp
        p = f"vit.{l}."
        add(p + "ln1.g", (d,), GAIN); add(p + "ln1.b", (d,), VEC)
        add(p + "wq", (d, d), MAT); add(p + "bq", (d,), VEC)
        add(p + "wk", (d, d), MAT); add(p + "bk", (d,), VEC)
        add(p + "wv", (d, d), MAT); add(p + "bv", (d,), VEC)
        add(p + "wo", (d, d), MAT); add(p + "bo", (d,), VEC)
        add(p + "ln2.g", (d,), GAIN); add(p + "ln2.b", (d,), VEC)
        add(p + "w1", (d, f), MAT); add(p + "b1", (f,), VEC)
        add(p + "w2", (f, d), MAT); add(p + "b2", (d,), VEC)
    if c.vit_layers > 0:
        add("vit.lnf.g", (c.vit_d,), GAIN); add("vit.lnf.b", (c.vit_d,), VEC)
        add("vit.proj.w", (c.vit_d * c.pix_shuffle ** 2, c.llm_d), MAT); add("vit.proj.b", (c.llm_d,), VEC)
    add("embed", (c.vocab, c.llm_d), VEC)
    D, Hq, Hk = c.llm_d, c.n_q * c.head_dim, c.n_kv * c.head_dim
    for l in range(c.llm_layers):
        p = f"llm.{l}."
        add(p + "ln1.g", (D,), GAIN)
        add(p + "wq", (D, Hq), MAT); add(p + "wk", (D, Hk), MAT); add(p + "wv", (D, Hk), MAT)
        add(p + "wo", (Hq, D), MAT)
        add(p + "ln2.g", (D,), GAIN)
        add(p + "wg", (D, c.llm_mlp), MAT); add(p + "wu", (D, c.llm_mlp), MAT)
        add(p + "wd", (c.llm_mlp, D), MAT)
    A, Da, Fa = c.action_dim, c.act_d, c.act_mlp
    if c.head_kind == HEAD_JOINT:
        add("act.in.w", (A, Da), MAT); add("act.in.b", (Da,), VEC)
        add("act.t1a.w", (Da, Da), MAT); add("act.t1t.w", (c.tdim, Da), MAT)
        add("act.t1.b", (Da,), VEC)
        add("act.t2.w", (Da, Da), MAT); add("act.t2.b", (Da,), VEC)
        for l in range(c.act_layers):
            p = f"act.{l}."
            add(p + "ln1.g", (Da,), GAIN)
            add(p + "wq", (Da, Hq), MAT); add(p + "wk", (Da, Hk), MAT); add(p + "wv", (Da, Hk), MAT)
            add(p + "wo", (Hq, Da), MAT)
            add(p + "ln2.g", (Da,), GAIN)
            add(p + "wg", (Da, Fa), MAT); add(p + "wu", (Da, Fa), MAT)
            add(p + "wd", (Fa, Da), MAT)
        add("act.lnf.g", (Da,), GAIN)
        add("act.out.w", (Da, A), MAT); add("act.out.b", (A,), VEC)
    else:
        # VLM -> DiT hand-off (runs in the VLM stage)
        add("llm.lnf.g", (D,), GAIN)
        add("vp.w", (D, Da), MAT); add("vp.b", (Da,), VEC)
        for l in range(c.act_layers):
            p = f"xkv.{l}."
            add(p + "wk", (Da, Da), MAT); add(p + "bk", (Da,), VEC)
            add(p + "wv", (Da, Da), MAT); add(p + "bv", (Da,), VEC)
        add("state.w", (c.state_dim, Da), MAT); add("state.b", (Da,), VEC)
        # DiT
        add("dit.t1.w", (c.tdim, Da), MAT); add("dit.t1.b", (Da,), VEC)
        add("dit.t2.w", (Da, Da), MAT); add("dit.t2.b", (Da,), VEC)
        add("dit.ain.w", (A, Da), MAT); add("dit.ain.b", (Da,), VEC)
        add("dit.pos", (c.horizon + 1, Da), VEC)
        for l in range(c.act_layers):
            p = f"dit.{l}."
            add(p + "mod.w", (Da, 6 * Da), MAT); add(p + "mod.b", (6 * Da,), VEC)
            add(p + "wq", (Da, Da), MAT); add(p + "bq", (Da,), VEC)
            add(p + "wk", (Da, Da), MAT); add(p + "bk", (Da,), VEC)
            add(p + "wv", (Da, Da), MAT); add(p + "bv", (Da,), VEC)
            add(p + "wo", (Da, Da), MAT); add(p + "bo", (Da,), VEC)
            add(p + "cq.w", (Da, Da), MAT); add(p + "cq.b", (Da,), VEC)
            add(p + "co.w", (Da, Da), MAT); add(p + "co.b", (Da,), VEC)
            add(p + "w1", (Da, Fa), MAT); add(p + "b1", (Fa,), VEC)
            add(p + "w2", (Fa, Da), MAT); add(p + "b2", (Da,), VEC)
        add("dit.modf.w", (Da, 2 * Da), MAT); add("dit.modf.b", (2 * Da,), VEC)
        add("dit.out.w", (Da, A), MAT); add("dit.out.b", (A,), VEC)
    return s


def weight_count(c: VLAConfig) -> int:
    return int(sum(int(np.prod(sh)) for _, sh, _ in weight_schema(c)))


def make_weights(c: VLAConfig, threads: int = 0) -> np.ndarray:
    """Flat fp32 parameter buffer in canonical order (seed 1000 + cfg.seed).
    Tensor i draws from its own stream, so tensors are filled by a thread
    pool (numpy releases the GIL while it draws) with the same values as a
    serial fill."""
    import concurrent.futures as cf
    import os
    sch = weight_schema(c)
    out = np.empty(weight_count(c), dtype=np.float32)
    offs, off = [], 0
    for _, shape, _ in sch:
        offs.append(off)
        off += int(np.prod(shape))

    def fill(i):
        _, shape, kind = sch[i]
        n = int(np.prod(shape))
        rng = np.random.Generator(np.random.PCG64(
            np.random.SeedSequence(1000 + c.seed, spawn_key=(i,))))
        v = out[offs[i]:offs[i] + n]
        rng.standard_normal(out=v, dtype=np.float32)
        v *= np.float32(0.02)
        if kind == GAIN:
            v += np.float32(1.0)

    nt = threads or min(16, os.cpu_count() or 1)
    if nt <= 1 or out.size < (1 << 22):
        for i in range(len(sch)):
            fill(i)
    else:
        # largest tensors first so the pool stays busy to the end
        order = sorted(range(len(sch)), key=lambda i: -int(np.prod(sch[i][1])))
        with cf.ThreadPoolExecutor(max_workers=nt) as ex:
            list(ex.map(fill, order))
    return out


def weight_views(c: VLAConfig, flat: np.ndarray) -> Dict[str, np.ndarray]:
    """Name -> view of the flat buffer with the tensor's shape."""
    views, off = {}, 0
    for name, shape, _ in weight_schema(c):
        n = int(np.prod(shape))
        views[name] = flat[off:off + n].reshape(shape)
        off += n
    assert off == flat.size, (off, flat.size)
    return views


# ---------------------------------------------------------------------------
# Request inputs (row r is identical for every batch size)
# ---------------------------------------------------------------------------
def _rows(base: int, rows, fn):
    out = []
    for r in rows:
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence(base, spawn_key=(int(r),))))
        out.append(fn(rng))
    return np.stack(out) if out else None


def make_pixels(c: VLAConfig, batch: int, first_row: int = 0) -> np.ndarray:
    """U[0,1) fp32 [B, n_img, 3, H, W] (stands in for camera frames)."""
    sh = (c.n_img, 3, c.img_hw, c.img_hw)
    return _rows(2000 + c.seed, range(first_row, first_row + batch),
                 lambda g: g.random(sh, dtype=np.float32)).reshape((batch,) + sh)


def make_text_ids(c: VLAConfig, batch: int, first_row: int = 0) -> np.ndarray:
    """U[0, vocab) int32 [B, n_text] (stands in for a tokenized instruction)."""
    return _rows(3000 + c.seed, range(first_row, first_row + batch),
                 lambda g: g.integers(0, c.vocab, size=(c.n_text,), dtype=np.int32)
                 ).reshape(batch, c.n_text).astype(np.int32)


def make_noise(c: VLAConfig, batch: int, first_row: int = 0) -> np.ndarray:
    """N(0,1) fp32 [B, horizon, action_dim]: the Euler loop's starting point."""
    sh = (c.horizon, c.action_dim)
    return _rows(4000 + c.seed, range(first_row, first_row + batch),
                 lambda g: g.standard_normal(sh, dtype=np.float32)).reshape((batch,) + sh)


def make_state(c: VLAConfig, batch: int, first_row: int = 0) -> np.ndarray:
    """N(0,1) fp32 [B, state_dim] proprioceptive state (DiT head only)."""
    return _rows(5000, range(first_row, first_row + batch),
                 lambda g: g.standard_normal((c.state_dim,), dtype=np.float32)
                 ).reshape(batch, c.state_dim)


def make_inputs(c: VLAConfig, batch: int, first_row: int = 0) -> Dict[str, np.ndarray]:
    d = {"pixels": make_pixels(c, batch, first_row),
         "text_ids": make_text_ids(c, batch, first_row),
         "noise": make_noise(c, batch, first_row)}
    if c.head_kind == HEAD_DIT:
        d["state"] = make_state(c, batch, first_row)
    return d


# ---------------------------------------------------------------------------
# Robot traffic for the serving workload
# ---------------------------------------------------------------------------
def poisson_arrivals(n_robots: int, rate_hz, duration_s: float, epoch: int,
                     n_models: int = 2) -> np.ndarray:
    """Arrival trace for ``n_robots`` robots, robot i -> model i % n_models,
    each with exponential inter-arrival gaps at its rate (Hz). Returns a
    structured array (t_ns int64, model int32, robot int32) sorted by time.
    Seed 6000 + epoch; robot r draws from its own spawn key."""
    rates = np.broadcast_to(np.asarray(rate_hz, dtype=np.float64), (n_robots,))
    ts, ms, rs = [], [], []
    for r in range(n_robots):
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(6000 + epoch, spawn_key=(r,))))
        t = 0.0
        while True:
            t += g.exponential(1.0 / rates[r])
            if t >= duration_s:
                break
            ts.append(int(t * 1e9)); ms.append(r % n_models); rs.append(r)
    out = np.zeros(len(ts), dtype=[("t_ns", np.int64), ("model", np.int32), ("robot", np.int32)])
    out["t_ns"], out["model"], out["robot"] = ts, ms, rs
    return np.sort(out, order=["t_ns", "robot"], kind="stable")


def periodic_arrivals(n_robots: int, rate_hz, duration_s: float, epoch: int,
                      n_models: int = 2) -> np.ndarray:
    """Paper's robot traffic model (Section 5.1): each robot starts at an offset
    drawn from U[0, 1/f) and then sends one request every 1/f seconds."""
    rates = np.broadcast_to(np.asarray(rate_hz, dtype=np.float64), (n_robots,))
    ts, ms, rs = [], [], []
    for r in range(n_robots):
        g = np.random.Generator(np.random.PCG64(np.random.SeedSequence(7000 + epoch, spawn_key=(r,))))
        per = 1.0 / rates[r]
        t = g.uniform(0.0, per)
        while t < duration_s:
            ts.append(int(t * 1e9)); ms.append(r % n_models); rs.append(r)
            t += per
    out = np.zeros(len(ts), dtype=[("t_ns", np.int64), ("model", np.int32), ("robot", np.int32)])
    out["t_ns"], out["model"], out["robot"] = ts, ms, rs
    return np.sort(out, order=["t_ns", "robot"], kind="stable")
