"""Decode-step model of the GPU tests: builds a model through the C ABI, runs traced
steps and checks every linear teacher-forced against the oracle.

Each linear's traced input is fed to the oracle linear; the oracle output, finished
with the same ReLU / residual sum in float64, must match the traced output within
2e-3 + the activation type's rounding.  Placement of the value slice and of the
ReLU output is checked bit for bit; the LayerNorm inputs are checked against the
oracle's LayerNorm.  For large shapes the oracle can be asked for sampled output
rows only (the same rows for every batch row).
"""
import numpy as np
import pytest

import oracle
import synth
from oracle import decode_step as ods
from common import TOL, U_ACT, Pinned, np_from_dev, rel_err, torch_dev_from_np

torch = pytest.importorskip("torch")
hg = pytest.importorskip("paper_2403_01164_amd")

NAMES = ("qkv", "out", "fc1", "fc2")


def shapes(H, F):
    return {"qkv": (3 * H, H), "out": (H, H), "fc1": (F, H), "fc2": (H, F)}


class Model:
    """weights: (W, b) lists of another Model to share its host weights (this model then
    does not free them)."""

    def __init__(self, ctx, L, H, F, dtype, alpha, resident, max_batch=8, seed=0, weights=None):
        self.ctx, self.L, self.H, self.F, self.dtype = ctx, L, H, F, dtype
        self.owns = weights is None
        self.W, self.b = ([], []) if weights is None else (list(weights[0]), list(weights[1]))
        for l in range(L if weights is None else 0):
            for name in NAMES:
                n, k = shapes(H, F)[name]
                W = Pinned(hg, ctx, (n, k), np.uint16)
                b = Pinned(hg, ctx, (n,), np.uint16)
                synth.fill_normal_ptr(W.ptr, n * k, dtype, seed, synth.weight_id(l, name), 0.0, 0.02)
                synth.fill_normal_ptr(b.ptr, n, dtype, seed, synth.bias_id(l, name), 0.0, 0.02)
                self.W.append(W)
                self.b.append(b)
        self.alpha = list(alpha) if hasattr(alpha, "__len__") else [alpha] * (4 * L)
        self.resident = list(resident) if hasattr(resident, "__len__") else [resident] * (4 * L)
        self.m = hg.hetegen_model_create(ctx, L, H, F, dtype, [w.ptr for w in self.W], [b.ptr for b in self.b],
                                         self.alpha, self.resident, max_batch)

    def step(self, x_bits, trace=False):
        B = x_bits.shape[0]
        x = torch_dev_from_np(x_bits)
        out = torch.full((B, self.H), -1, dtype=torch.int16, device="cuda")
        tr = None
        if trace:
            nb = hg.hetegen_model_trace_bytes(self.m, B)
            tr = torch.full((nb // 2,), -1, dtype=torch.int16, device="cuda")
            hg.hetegen_model_set_trace(self.m, tr.data_ptr(), nb)
        s = torch.cuda.current_stream().cuda_stream
        hg.hetegen_decode_step(self.ctx, self.m, x.data_ptr(), out.data_ptr(), B, s)
        torch.cuda.synchronize()
        if trace:
            hg.hetegen_model_set_trace(self.m, 0, 0)
        o = np_from_dev(out, np.uint16)
        return (o, np_from_dev(tr, np.uint16)) if trace else o

    def split_trace(self, tr, B):
        items, off = [], 0
        for l in range(self.L):
            for name in NAMES:
                n, k = shapes(self.H, self.F)[name]
                xin = tr[off:off + B * k].reshape(B, k)
                off += B * k
                yout = tr[off:off + B * n].reshape(B, n)
                off += B * n
                items.append((name, l, xin, yout))
        return items

    def step_kv(self, x_bits, pos, trace=False):
        B = x_bits.shape[0]
        x = torch_dev_from_np(x_bits)
        out = torch.full((B, self.H), -1, dtype=torch.int16, device="cuda")
        tr = None
        if trace:
            nb = hg.hetegen_model_trace_bytes(self.m, B)
            tr = torch.full((nb // 2,), -1, dtype=torch.int16, device="cuda")
            hg.hetegen_model_set_trace(self.m, tr.data_ptr(), nb)
        s = torch.cuda.current_stream().cuda_stream
        hg.hetegen_decode_step_kv(self.ctx, self.m, x.data_ptr(), out.data_ptr(), B, pos, s)
        torch.cuda.synchronize()
        if trace:
            hg.hetegen_model_set_trace(self.m, 0, 0)
        o = np_from_dev(out, np.uint16)
        return (o, np_from_dev(tr, np.uint16)) if trace else o

    def check_teacher_forced(self, x_bits, tr, attn=None, sample=None):
        """sample: None checks every output; n > 0 checks, per linear, the first and last
        8 output rows and n more drawn at random (fixed seed), for every batch row."""
        dt, H = self.dtype, self.H
        B = x_bits.shape[0]
        items = self.split_trace(tr, B)
        x_l = x_bits
        worst = 0.0
        rng = np.random.default_rng(1234)
        for i, (name, l, xin, yout) in enumerate(items):
            W, b = self.W[i].a, self.b[i].a
            N = W.shape[0]
            if sample is None or N <= 16 + sample:
                cols = np.arange(N)
                lin = oracle.linear(xin, W, b, dt).astype(np.float64)
            else:
                cols = np.unique(np.concatenate([np.arange(8), np.arange(N - 8, N),
                                                 rng.choice(N, size=sample, replace=False)]))
                rb = np.repeat(np.arange(B), cols.size)
                rj = np.tile(cols, B)
                lin = oracle.linear_sample(xin, W, b, dt, rb, rj).astype(np.float64).reshape(B, cols.size)
            got = oracle.decode(yout, dt)[:, cols]
            if name == "qkv":
                h_ref = ods.layer_norm(oracle.decode(x_l, dt))
                assert rel_err(oracle.decode(xin, dt), h_ref) <= TOL + U_ACT[dt], ("LN", l)
                ref = lin
                qkv_out = yout
            elif name == "out":
                if attn is None:
                    assert np.array_equal(xin, qkv_out[:, 2 * H:3 * H]), ("V slice", l)
                else:  # attention over the cache, from the traced q | k | v
                    e = rel_err(oracle.decode(xin, dt), attn(l, qkv_out))
                    assert e <= TOL + U_ACT[dt], ("attention", l, e)
                ref = oracle.decode(x_l, dt).astype(np.float64)[:, cols] + lin
                x_mid = yout
            elif name == "fc1":
                h_ref = ods.layer_norm(oracle.decode(x_mid, dt))
                assert rel_err(oracle.decode(xin, dt), h_ref) <= TOL + U_ACT[dt], ("LN2", l)
                ref = np.maximum(lin, 0.0)
                f_out = yout
            else:
                assert np.array_equal(xin, f_out), ("fc2 input", l)
                ref = oracle.decode(x_mid, dt).astype(np.float64)[:, cols] + lin
                x_l = yout
            e = rel_err(got, ref)
            worst = max(worst, e)
            assert e <= TOL + U_ACT[dt], (name, l, e)
        return x_l, worst

    def free(self):
        hg.hetegen_model_destroy(self.ctx, self.m)
        if self.owns:
            for p in self.W + self.b:
                p.free()


