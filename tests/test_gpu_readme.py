"""The usage example of README.md runs as written: its python block is
executed after a prelude that defines the names it leaves to the reader
(a generated group of rollouts, the trunk's hidden states, the LM head, the
histograms), and its outputs are checked for shape and sense."""

import os
import re

import numpy as np
import pytest
import torch

from conftest import ROOT
from gpu_util import require_gpu

pytestmark = pytest.mark.gpu


def _example():
    text = open(os.path.join(ROOT, "README.md")).read()
    blocks = re.findall(r"```python\n(.*?)```", text, re.S)
    assert blocks, "README.md has no python block"
    return blocks[0]


def test_readme_usage_example_runs():
    require_gpu()
    rng = np.random.default_rng(0)
    G, n_groups = 4, 8
    n_new = G * n_groups
    lens = rng.integers(100, 400, n_new).astype(np.int32)
    total = int(lens.sum())
    T, d, V, n_draw = 2048, 128, 1000, 16
    env = {
        "group_off": torch.arange(0, n_new + 1, G, dtype=torch.int32, device="cuda"),
        "lengths": torch.from_numpy(lens).cuda(),
        "src_off": torch.from_numpy(np.concatenate([[0], np.cumsum(lens)[:-1]])).cuda(),
        "rewards": torch.from_numpy((rng.random(n_new) < 0.5).astype(np.float32)).cuda(),
        "version": 3,
        "tokens": torch.from_numpy(rng.integers(0, V, total).astype(np.int32)).cuda(),
        "old_logp": torch.from_numpy((-rng.random(total) * 5).astype(np.float32)).cuda(),
        "step": 0, "n_draw": n_draw, "T": T, "d": d, "V": V, "n_seq_total": n_draw,
        "hidden": torch.randn(T, d, device="cuda").to(torch.bfloat16),
        "W": (torch.randn(V, d, device="cuda") * 0.02).to(torch.bfloat16),
        "dW": torch.zeros(V, d, device="cuda"),
        "age_hist": torch.zeros(8, dtype=torch.int64, device="cuda"),
        "since_hist": torch.zeros(8, dtype=torch.int64, device="cuda"),
    }
    print("[readme] running the usage example", flush=True)
    exec(compile(_example(), "README.md", "exec"), env)
    torch.cuda.synchronize()
    b = env["b"]
    assert int(b["n_tokens"].item()) == T  # 16 draws of >= 100 tokens fill the window
    assert torch.isfinite(env["loss"]).all() and torch.isfinite(env["dlogp"]).all()
    assert torch.isfinite(env["dhidden"]).all() and torch.isfinite(env["dW"]).all()
    assert int(env["age_hist"].sum().item()) == n_draw
    assert int(env["since_hist"].sum().item()) == n_draw
    assert env["ring"].n_live == n_new
