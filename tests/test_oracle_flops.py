"""Pins for the oracle's FLOP accounting of realised token trajectories
(App. E.4; actor architecture App. A.1; grids Table 3).  CPU only.

The count is pinned to torch's own FLOP counter (FlopCounterMode: two FLOPs
per multiply-accumulate of every matmul / linear / convolution) run on
meta-device modules of the stated architecture along the same trajectories,
and to the Native GFLOPs of Table 1 within the share of operations the paper
counts beyond multiply-accumulates (its figures are 0.2-0.4 % higher).
"""
import math

import numpy as np
import pytest
import torch
from torch import nn
from torch.utils.flop_counter import FlopCounterMode

import oracle

META = torch.device("meta")


class Block(nn.Module):
    """Pre-LN Transformer block; attention over all n tokens, then the rows
    past m are dropped before the MLP (the pruning operator, Eq. (1))."""

    def __init__(self, d, heads, r):
        super().__init__()
        self.h = heads
        self.ln1, self.ln2 = nn.LayerNorm(d), nn.LayerNorm(d)
        self.qkv, self.proj = nn.Linear(d, 3 * d), nn.Linear(d, d)
        self.fc1, self.fc2 = nn.Linear(d, r * d), nn.Linear(r * d, d)

    def forward(self, x, m):
        n, d = x.shape[1], x.shape[2]
        qkv = self.qkv(self.ln1(x)).reshape(1, n, 3, self.h, d // self.h).permute(2, 0, 3, 1, 4)
        q, k, v = qkv[0], qkv[1], qkv[2]
        a = torch.softmax(torch.matmul(q, k.transpose(-2, -1)), dim=-1)
        o = torch.matmul(a, v).transpose(1, 2).reshape(1, n, d)
        x = (x + self.proj(o))[:, :m]
        return x + self.fc2(nn.functional.gelu(self.fc1(self.ln2(x))))


class Actor(nn.Module):
    def __init__(self, d, M):
        super().__init__()
        self.gate = nn.Sequential(nn.Linear(d + 19, 64), nn.SiLU(), nn.Linear(64, 1))
        self.w_in, self.w_h = nn.Linear(d, 128), nn.Linear(3, 128)
        self.enc = Block(128, 4, 2)
        self.budget = nn.Sequential(nn.LayerNorm(128), nn.Linear(128, 128), nn.GELU(), nn.Linear(128, M))
        self.w_k = nn.Linear(1, 128)
        self.sel = nn.Sequential(nn.Linear(128, 64), nn.SiLU(), nn.Linear(64, 1))

    def run_gate(self, kcls):
        return self.gate(torch.cat([kcls, torch.zeros(1, 19, device=META)], dim=1))

    def run_controller(self, keys):
        n = keys.shape[1]
        x = self.w_in(keys)
        x = torch.cat([x[:, :1] + self.w_h(torch.zeros(1, 1, 3, device=META)), x[:, 1:]], dim=1)
        z = self.enc(x, n)
        self.budget(z[:, 0])
        self.sel(z[:, 1:] + self.w_k(torch.zeros(1, 1, 1, device=META)))


def torch_count(T, d, heads, L, N0, patch, M, head_inputs, actor):
    """FLOPs torch counts for one image along the trajectory T [L+1]."""
    side = int(round(math.sqrt(N0))) * patch
    embed = nn.Conv2d(3, d, patch, patch, device=META)
    blocks = [Block(d, heads, 4).to(META) for _ in range(1)]      # one set of weights; shapes are what count
    head = nn.Linear(head_inputs * d, 1000, device=META)
    act = Actor(d, M).to(META)
    with FlopCounterMode(display=False) as fc:
        x = embed(torch.zeros(1, 3, side, side, device=META)).flatten(2).transpose(1, 2)
        x = torch.cat([torch.zeros(1, 1, d, device=META), x], dim=1)
        for l in range(L):
            n, m = int(T[l]), int(T[l + 1])
            keys = torch.zeros(1, n, d, device=META)
            if actor and n - 1 >= 6:
                act.run_gate(keys[:, 0])
            if actor and m < n:
                act.run_controller(keys)
            x = blocks[0](x[:, :n], m)
        head(torch.zeros(1, head_inputs * d, device=META))
    return fc.get_total_flops()


def legal_trajectory(rng, L, N0, M):
    T = [N0 + 1]
    for _ in range(L):
        nv = T[-1] - 1
        legal = [k for k in range(2, 2 * M + 1, 2) if k <= nv - 4]
        k = int(rng.choice(legal)) if legal and rng.random() < 0.5 else 0
        T.append(T[-1] - k)
    return np.array(T)


BACKBONES = {  # d, heads, L, N0, patch, head inputs (Table 3; DINOv2's LC1 readout doubles the head input)
    "DeiT-B": (768, 12, 12, 196, 16, 1, 35.2),
    "ViT-B": (768, 12, 12, 196, 16, 1, 35.2),
    "ViT-L": (1024, 16, 24, 196, 16, 1, 123.4),
    "DINOv2-B/14": (768, 12, 12, 256, 14, 2, 46.5),
}


@pytest.mark.parametrize("name", list(BACKBONES))
def test_native_matches_torch_counter_and_table1(name):
    d, h, L, N0, p, hi, printed = BACKBONES[name]
    M = (N0 - 4) // 2
    T = np.full((L + 1, 1), N0 + 1)
    ours = int(oracle.trajectory_flops(T, d, L, N0, p, M, head_inputs=hi, actor=False)[0])
    assert ours == torch_count(T[:, 0], d, h, L, N0, p, M, hi, actor=False)
    gap = (printed - ours / 1e9) / printed
    assert 0 < gap < 0.005, (name, ours / 1e9, printed)


@pytest.mark.parametrize("name", ["DeiT-B", "ViT-L", "DINOv2-B/14"])
def test_pruned_trajectories_with_actor_match_torch_counter(name):
    d, h, L, N0, p, hi, _ = BACKBONES[name]
    M = (N0 - 4) // 2
    rng = np.random.default_rng(len(name))
    T = np.stack([legal_trajectory(rng, L, N0, M) for _ in range(3)], axis=1)
    T[:, 0] = N0 + 1                                     # one image never pruned
    ours = oracle.trajectory_flops(T, d, L, N0, p, M, head_inputs=hi, actor=True)
    for b in range(T.shape[1]):
        assert int(ours[b]) == torch_count(T[:, b], d, h, L, N0, p, M, hi, actor=True), b


def test_pruning_never_adds_flops_beyond_the_actor():
    d, h, L, N0, p, hi, _ = BACKBONES["DeiT-B"]
    M = (N0 - 4) // 2
    rng = np.random.default_rng(3)
    T = np.stack([legal_trajectory(rng, L, N0, M) for _ in range(50)], axis=1)
    backbone = oracle.trajectory_flops(T, d, L, N0, p, M, actor=False)
    native = oracle.trajectory_flops(np.full((L + 1, 1), N0 + 1), d, L, N0, p, M, actor=False)[0]
    assert np.all(backbone <= native)
    assert np.all((backbone < native) == np.any(np.diff(T, axis=0) < 0, axis=0))


def _battery():
    """True when the (possibly patched) oracle agrees with torch's counter on
    a native and a pruned DeiT-B trajectory and on a pruned DINOv2 one."""
    for name in ("DeiT-B", "DINOv2-B/14"):
        d, h, L, N0, p, hi, _ = BACKBONES[name]
        M = (N0 - 4) // 2
        T = np.stack([np.full(L + 1, N0 + 1), legal_trajectory(np.random.default_rng(9), L, N0, M)], axis=1)
        ours = oracle.trajectory_flops(T, d, L, N0, p, M, head_inputs=hi, actor=True)
        for b in range(2):
            if int(ours[b]) != torch_count(T[:, b], d, h, L, N0, p, M, hi, actor=True):
                return False
    return True


def _mlp_on_attention_tokens(tokens, *a, **k):
    T = np.asarray(tokens)
    return oracle_trajectory(np.vstack([T[:1], T[:-1]]), *a, **k)


oracle_trajectory = oracle.trajectory_flops
FLOP_MUTANTS = {
    "one_attention_product": ("_attention_block_macs",
                              lambda n, d, r: (n * d * 3 * d + n * n * d + n * d * d, d * r * d + r * d * d)),
    "mlp_ratio_two": ("_attention_block_macs",
                      lambda n, d, r: (n * d * 3 * d + 2 * n * n * d + n * d * d, 2 * d * d + 2 * d * d)),
    "gate_without_history": ("actor_gate_macs", lambda d, **k: (d + 16) * 64 + 64),
    "no_selector": ("actor_controller_macs",
                    lambda n, d, M, **k: n * d * 128 + 3 * 128 + 3 * n * 128 * 128 + 2 * n * n * 128
                    + n * 128 * 128 + 2 * n * 128 * 256 + 128 * 128 + 128 * M),
    "mlp_on_attention_tokens": ("trajectory_flops", _mlp_on_attention_tokens),
}


def test_unmodified_flop_oracle_passes():
    assert _battery()


@pytest.mark.parametrize("name", sorted(FLOP_MUTANTS))
def test_flop_mutant_is_caught(monkeypatch, name):
    attr, fn = FLOP_MUTANTS[name]
    monkeypatch.setattr(oracle, attr, fn)
    assert not _battery(), f"planted mistake '{name}' passed the torch-counter pin"
