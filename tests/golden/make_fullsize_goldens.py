"""Write the oracle's expected outputs for the full-size pi0-shaped and
GR00T-like models (test infrastructure; calls only the oracle and the seeded
generators).

    python tests/golden/make_fullsize_goldens.py [pi0] [gr00t]

For each model, rows 0 and max_batch-1 of the seeded request inputs go
through the fp64 oracle (bf16-rounded parameters). Batch rows are
independent, so the same values serve a batch-1 run of row 0 and both rows of
a max-batch run. Stored (numpy .npz, float32 values of the fp64 results):

* ``actions`` [2, horizon, action_dim] and ``noise`` [2, horizon, action_dim];
* joint head: ``k``/``v`` [2, layers, n_kv, 3, head_dim], the post-RoPE
  prefix keys and values at positions ``kv_pos`` (first, middle, last);
* DiT head: ``kc``/``vc`` [2, layers, 3, act_d] at ``kv_pos`` and ``state``
  [2, act_d];
* ``weights_probe``: parameter count and sums of the first and last 4096
  parameters, so a test can tell whether the generators still produce the
  parameters these values were computed from.

Memory: the parameters stay in one fp32 buffer (bf16-rounded) and each
tensor is upcast to fp64 when the oracle reads it, so a pi0-shaped model
needs ~12 GB of host memory rather than ~22 GB for an fp64 copy.
"""
from __future__ import annotations

import os
import sys
import time

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(os.path.dirname(HERE))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

from oracle import vla as O  # noqa: E402
from paper_2609_12075_amd import synth as S  # noqa: E402


class Fp64Views(dict):
    """Name -> fp64 copy of a tensor, made when the oracle reads it."""

    def __init__(self, views):
        super().__init__()
        self._views = views

    def __getitem__(self, k):
        return self._views[k].astype(np.float64)

    def __contains__(self, k):
        return k in self._views

    def keys(self):
        return self._views.keys()


def golden_path(name: str) -> str:
    return os.path.join(HERE, f"fullsize_{name}.npz")


def weights_probe(flat: np.ndarray) -> np.ndarray:
    return np.array([flat.size, float(flat[:4096].astype(np.float64).sum()),
                     float(flat[-4096:].astype(np.float64).sum())])


def make(name: str) -> None:
    cfg = S.CONFIGS[name]
    t0 = time.time()
    flat = S.make_weights(cfg)
    probe = weights_probe(flat)
    for chunk in range(0, flat.size, 1 << 26):        # bf16 rounding in place, chunk by chunk
        flat[chunk:chunk + (1 << 26)] = O.bf16_round(flat[chunk:chunk + (1 << 26)])
    W = Fp64Views(S.weight_views(cfg, flat))
    rows = [0, cfg.max_batch - 1]
    per_row = [S.make_inputs(cfg, 1, first_row=r) for r in rows]
    inp = {k: np.concatenate([d[k] for d in per_row]) for k in per_row[0]}
    print(f"[{name}] parameters ready in {time.time() - t0:.1f} s", flush=True)
    P = cfg.prefix_len
    kv_pos = np.array([0, P // 2, P - 1])
    out = {"rows": np.array(rows), "kv_pos": kv_pos, "weights_probe": probe}
    acts, ks, vs, kcs, vcs, sts = [], [], [], [], [], []
    for i in range(len(rows)):
        t1 = time.time()
        st = inp["state"][i] if "state" in inp else None
        pre = O.prefill_row(cfg, W, inp["pixels"][i], inp["text_ids"][i], st)
        act = O.denoise_row(cfg, W, pre, inp["noise"][i], cfg.steps)
        acts.append(act)
        if cfg.head_kind == S.HEAD_JOINT:
            ks.append(np.stack([k[:, kv_pos, :] for k in pre["k"]]))
            vs.append(np.stack([v[:, kv_pos, :] for v in pre["v"]]))
        else:
            kcs.append(np.stack([k[kv_pos] for k in pre["kc"]]))
            vcs.append(np.stack([v[kv_pos] for v in pre["vc"]]))
            sts.append(pre["state"])
        print(f"[{name}] row {rows[i]}: {time.time() - t1:.1f} s", flush=True)
    out["actions"] = np.stack(acts).astype(np.float32)
    out["noise"] = inp["noise"].astype(np.float32)
    if ks:
        out["k"], out["v"] = np.stack(ks).astype(np.float32), np.stack(vs).astype(np.float32)
    else:
        out["kc"], out["vc"] = np.stack(kcs).astype(np.float32), np.stack(vcs).astype(np.float32)
        out["state"] = np.stack(sts).astype(np.float32)
    np.savez_compressed(golden_path(name), **out)
    print(f"[{name}] wrote {golden_path(name)} ({os.path.getsize(golden_path(name)) / 1e3:.0f} kB) "
          f"in {time.time() - t0:.1f} s", flush=True)


if __name__ == "__main__":
    for n in (sys.argv[1:] or ["pi0", "gr00t"]):
        make(n)
