"""Helpers for the GPU parity tests (imported by tests only)."""

import numpy as np
import pytest
import torch


def require_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")
    import paper_2604_08706_amd as rbp  # raises if librbpolicy.so is missing
    rbp.lib()
    return rbp


def rel_l2(a, b):
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    den = np.linalg.norm(b)
    return np.linalg.norm(a - b) / (den if den > 0 else 1.0)


def to_np(t):
    return t.detach().cpu().numpy()


def bf16_to_f64(t):
    return t.detach().cpu().to(torch.float64).numpy()


class DeviceRing:
    """A FIFO record table uploaded as a device ring buffer.

    Logical slot s lives in physical row (head + s) % capacity; rows that hold
    no live record get junk values (they must never be read)."""

    def __init__(self, rbp, length, arena_off, reward, advantage, version, arena_tok,
                 arena_old, head=0, capacity=None):
        n = len(length)
        cap = n if capacity is None else capacity
        assert n <= cap
        phys = (head + np.arange(n)) % cap

        def ring(vals, dtype, junk):
            a = np.full(cap, junk, dtype=dtype)
            a[phys] = np.asarray(vals, dtype=dtype)
            return torch.from_numpy(a).cuda()

        self.t_len = ring(length, np.int32, 7)
        self.t_off = ring(arena_off, np.int64, 0)
        self.t_rew = ring(reward, np.float32, 1.0)
        self.t_adv = ring(advantage, np.float32, 123.0)
        self.t_ver = ring(version, np.int32, -99)
        self.t_tok = arena_tok if isinstance(arena_tok, torch.Tensor) else \
            torch.from_numpy(np.asarray(arena_tok, dtype=np.int32)).cuda()
        self.t_old = arena_old if isinstance(arena_old, torch.Tensor) else \
            torch.from_numpy(np.asarray(arena_old, dtype=np.float32)).cuda()
        self.rec = rbp.make_records(n, cap, head, self.t_off, self.t_len, self.t_rew,
                                    self.t_adv, self.t_ver, self.t_tok, self.t_old)
        self.capacity = cap
