"""The seeded workload generators: shapes, determinism, storage rounding, and
that they stay independent of both the oracle and the GPU package."""

import ast
import os

import numpy as np
import pytest
import torch

import workloads as W
from oracle import decode, prefill

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _imports(path):
    tree = ast.parse(open(path).read())
    names = set()
    for node in ast.walk(tree):
        if isinstance(node, ast.Import):
            names |= {a.name.split(".")[0] for a in node.names}
        elif isinstance(node, ast.ImportFrom) and node.module:
            names.add(node.module.split(".")[0])
    return names


def test_generators_and_oracle_are_independent():
    gen = _imports(os.path.join(ROOT, "workloads", "__init__.py"))
    assert "oracle" not in gen and "paper_2608_00528_amd" not in gen
    for f in os.listdir(os.path.join(ROOT, "oracle")):
        if f.endswith(".py"):
            imp = _imports(os.path.join(ROOT, "oracle", f))
            assert "workloads" not in imp and "paper_2608_00528_amd" not in imp and "torch" not in imp


def test_config_shapes():
    c = W.CONFIGS
    assert c["llama8b_128k"].L == 131068 and c["llama8b_128k"].R == 160 and c["llama8b_128k"].G == 4
    assert c["qwen7b_128k"].Dp == 512 and c["qwen7b_128k"].G == 7
    assert c["tiny_fp32"].R == 64 and c["tiny_fp32"].dtype == "fp32"
    assert c["llama8b_32L_sustained"].layers == 32 and c["llama8b_32L_sustained"].steps == 256


def test_latent_state_deterministic_and_rounded():
    wl = W.CONFIGS["llama8b_32k"].scaled(N=2048, batch=2)
    a = W.latent_state(wl, seed=3)
    b = W.latent_state(wl, seed=3)
    for k in ("coef_k", "bases_v", "q", "sink_k"):
        assert np.array_equal(a[k], b[k])
    assert np.array_equal(W.round_storage(a["coef_k"], "bf16"), a["coef_k"])
    c = W.latent_state(wl, seed=4)
    assert not np.array_equal(a["coef_k"], c["coef_k"])
    # capacity rows past L are zero
    d = W.latent_state(wl, seed=3, capacity=wl.L + 40)
    assert np.all(d["coef_k"][:, wl.L:] == 0) and np.array_equal(d["coef_k"][:, :wl.L], a["coef_k"])


@pytest.mark.parametrize("name", ["tiny_fp32", "llama8b_32k"])
def test_needles_are_recalled(name):
    """Sanity of the recipe, not parity: planted needles land in the index set."""
    wl = W.CONFIGS[name]
    if name != "tiny_fp32":
        wl = wl.scaled(N=8192)
    raw = W.raw_kv(wl, seed=0)
    st = prefill.prefill(raw["S_k"], raw["S_v"], wl.n_sink, wl.rank, wl.basis_groups,
                         center=True, dtype=wl.dtype)
    cfg = dict(n_kv_heads=wl.n_kv_heads, window=wl.window, topk=wl.topk, pool_kernel=7,
               rope_theta=wl.rope_theta, dtype=wl.dtype)
    r = decode.decode_step(cfg, wl.L, raw["q"], st["sink_k"], st["sink_v"], st["bases_k"],
                           st["bases_v"], st["coef_k"], st["coef_v"])
    assert np.isin(raw["needles"][0], r["idx"][0]).mean() >= 0.9


def test_sustained_layer_recipe():
    wl = W.CONFIGS["llama8b_32L_sustained"].scaled(batch=2, N=1024 + 4)
    L0, cap, T = wl.L - 1, 1040, 3
    a = W.sustained_layer(wl, 0, 5, L0, cap, T, device="cpu")
    b = W.sustained_layer(wl, 0, 5, L0, cap, T, device="cpu")
    other = W.sustained_layer(wl, 0, 6, L0, cap, T, device="cpu")
    for k in a:
        assert torch.equal(a[k], b[k]), k
    assert not torch.equal(a["coef_k"], other["coef_k"])
    assert a["coef_k"].shape == (2, cap, wl.R) and a["q"].shape == (T, 2, wl.n_q_heads, wl.head_dim)
    assert a["k_new"].shape == (T, 2, wl.Dp) and a["bases_v"].shape == (2, 1, wl.Dp, wl.rank)
    assert torch.count_nonzero(a["coef_k"][:, L0:]) == 0
    bk = a["bases_k"][0, 0].double()
    assert (bk.T @ bk - torch.eye(wl.rank, dtype=torch.float64)).abs().max() < 2e-2   # orthonormal up to bf16
    assert not torch.equal(a["bases_k"][0], a["bases_k"][1])                          # per-sequence bases
    norms = a["coef_k"][:, :L0].double().norm(dim=-1)
    assert 0.8 * np.sqrt(wl.Dp) < norms.mean() < 1.2 * np.sqrt(wl.Dp)
