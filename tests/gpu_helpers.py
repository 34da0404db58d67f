"""Helpers shared by the GPU parity tests: moving seeded inputs to the device and back,
and the relative L2 metric used for every floating-point comparison."""
import sys

import numpy as np

import synth


def log(msg):
    """Name the case on stdout before a GPU step (flushed, so it survives a crash)."""
    print(f"[gpu-case] {msg}", flush=True)
    sys.stdout.flush()


def dev(t):
    import torch
    if isinstance(t, synth.Tensor):
        if t.dtype == "bf16":
            return torch.from_numpy(np.ascontiguousarray(t.data).view(np.int16)).view(torch.bfloat16).cuda()
        return torch.from_numpy(np.ascontiguousarray(t.data)).cuda()
    a = np.asarray(t)
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()


def host(x):
    """Device tensor -> float64 numpy (exact widening of bf16/fp32)."""
    import torch
    return x.detach().to(torch.float32).cpu().numpy().astype(np.float64)


def rel_l2(got, ref):
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    return float(np.linalg.norm(got - ref) / max(np.linalg.norm(ref), 1e-300))


def workspace(nbytes):
    import torch
    # 256-byte aligned by the caching allocator
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device="cuda")
