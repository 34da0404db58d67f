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


def block_exp_index(M, nb, lde):
    """Byte index of each 64-column block's exponent in the library's block-scaled layout
    (per pair of blocks all rows in order, 4 bytes per row): block kb of row m at
    (kb // 2) * lde + 4 m + kb % 2.  Returns [M, nb] int64."""
    import numpy as np
    kb = np.arange(nb)
    return (kb // 2 * lde + kb % 2)[None, :] + 4 * np.arange(M)[:, None]


def check_block_output(codes, exps_buf, x_bf16, lde, pad=0xAB):
    """Codes [M, N] (uint8 device tensor) and the exponent buffer against the oracle's
    64-element MX quantization of the bf16 values x [M, N] (float64 host), bit for bit;
    the exponent buffer's other bytes must still hold pad."""
    import numpy as np
    import oracle
    import torch
    M, N = x_bf16.shape
    q, e = oracle.fp8.quantize_mx(x_bf16, 64)
    got = codes.view(torch.float8_e4m3fn).to(torch.float64).cpu().numpy().reshape(M, N)
    assert np.array_equal(got, q), "codes differ"
    buf = exps_buf.cpu().numpy()
    idx = block_exp_index(M, N // 64, lde)
    assert np.array_equal(buf[idx].astype(np.int64) - 127, e), "exponents differ"
    used = np.zeros(buf.size, bool)
    used[idx.ravel()] = True
    assert np.all(buf[~used] == pad), "bytes outside the exponents were written"
