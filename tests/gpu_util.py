"""Shared helpers of the GPU tests: build a handle from a synthetic workload,
move inputs to the device, and compare with the oracle."""
import numpy as np

import synth


def torch_mod():
    import torch
    return torch


def dev_prefix(w, k, v):
    """Prefix K/V as device tensors in the workload's storage type."""
    torch = torch_mod()
    if w.dtype == synth.BF16:
        kk = torch.from_numpy(synth.bf16_bits(k).view(np.int16)).cuda()
        vv = torch.from_numpy(synth.bf16_bits(v).view(np.int16)).cuda()
    else:
        kk = torch.from_numpy(np.ascontiguousarray(k)).cuda()
        vv = torch.from_numpy(np.ascontiguousarray(v)).cuda()
    return kk, vv


def dev(x):
    torch = torch_mod()
    return torch.from_numpy(np.array(x, dtype=np.float32)).cuda()  # a writable copy


def host(t):
    torch = torch_mod()
    torch.cuda.synchronize()
    return t.detach().cpu().numpy()


class Case:
    """A workload's inputs on host and device plus an open handle."""

    def __init__(self, w, seed=0, weights=None, noise_seed=0, max_batch=None, lens=None):
        from paper_2608_27384_amd.flashvla import Expert
        torch = torch_mod()
        self.w = w
        self.W = weights if weights is not None else synth.make_weights(w, seed)
        self.k, self.v, self.lens = synth.make_prefix(w, seed)
        if lens is not None:  # explicit prefix lengths (rows past them are never visible)
            self.lens = np.asarray(lens, dtype=np.int32)
            assert self.lens.shape == (w.batch,) and self.lens.max() <= w.max_prefix
        self.x = synth.make_buffer(w, seed)
        self.t = synth.noise_levels_batched(w)
        self.noise_seed = noise_seed
        self.ex = Expert(self.W, w, max_batch or w.batch, w.max_prefix, noise_seed)
        self.kd, self.vd = dev_prefix(w, self.k, self.v)
        self.ex.set_prefix(self.kd, self.vd, self.lens)
        self.xd = dev(self.x)
        self.td = dev(self.t)
        self.vout = torch.empty_like(self.xd)
        self.out = torch.empty((w.batch, w.chunk_len, w.action_dim), dtype=torch.float32,
                               device="cuda")

    def gpu_velocity(self, x=None):
        xd = self.xd if x is None else dev(x)
        self.ex.velocity(xd, self.td, self.vout)
        return host(self.vout)

    def oracle_velocity(self, b, x=None):
        import oracle
        x = self.x if x is None else x
        return oracle.velocity(x[b], self.t[b], self.k[:, b], self.v[:, b], int(self.lens[b]),
                               self.W, self.w)

    def close(self):
        self.ex.close()


def rel_err(got, ref):
    """max |got - ref| / max |ref| over one slice."""
    return float(np.max(np.abs(got - ref)) / max(np.max(np.abs(ref)), 1e-30))


def tol(w):
    return 1e-2 if w.dtype == synth.BF16 else 1e-4
