"""Seeded DiT block and step cases, run through the C ABI and through the fp64 oracle.

Both sides start from the same synth tensors; each computes its own positions (the
library's wam_chunk_positions/wam_rope_tables on the GPU side, oracle.chunk_positions
on the oracle side)."""
import numpy as np

import oracle
import synth
from gpu_helpers import dev, host, workspace


def lib():
    import paper_2602_15922_amd as w
    return w


def dims_of(wl, n_layers):
    return lib().make_dims(wl.d, wl.H, wl.Dh, wl.ffn, n_layers, wl.latent_ch, wl.act_dim, wl.text_dim,
                           wl.freq_dim, wl.eps)


def f64(params):
    return {k: v.f64 for k, v in params.items()}


def gpu_rope_tables(wl, B=None):
    w = lib()
    pos = w.wam_chunk_positions(wl.n_cached, wl.F, wl.Hg, wl.Wg, wl.A)
    cos, sin = w.wam_rope_tables(pos, wl.Dh)
    return dev(cos), dev(sin)


def oracle_positions(wl):
    return oracle.chunk_positions(wl.n_cached, wl.F, wl.Hg, wl.Wg, wl.A)


def prev_chunk_ids(wl):
    return np.repeat(np.arange(wl.n_cached), wl.L)


def upload_cache(wl, kc, vc, B):
    """[B, Lcap, H, Dh] device caches with the cached rows filled."""
    import torch
    k = torch.zeros((B, wl.Lcap, wl.H, wl.Dh), dtype=torch.bfloat16, device="cuda")
    v = torch.zeros_like(k)
    if kc is not None:
        k[:, :wl.cache_rows] = dev(kc)
        v[:, :wl.cache_rows] = dev(vc)
    return k, v


# ------------------------------------------------------------------------------ block
def fp8_caches(kcs, vcs, rows):
    """E4M3 code caches of bf16 caches [B, Lcap, H, 128] through the library's quantizers:
    K in 32-dim blocks (int32 exponent words [B, Lcap, H]), V with one scale per layer,
    max|V| / 448 over rows [0, rows).  Returns (k8s, kes, v8s, v_scales)."""
    import torch
    w = lib()
    k8s, kes, v8s, vsc = [], [], [], []
    for kc, vc in zip(kcs, vcs):
        Bc, Lcap, H, Dh = kc.shape
        k8 = torch.empty((Bc, Lcap, H, Dh), dtype=torch.uint8, device="cuda")
        ke = torch.empty((Bc, Lcap, H), dtype=torch.int32, device="cuda")
        w.wam_quantize_mx_fp8(kc.view(Bc * Lcap, H * Dh), k8.view(Bc * Lcap, H * Dh),
                              ke.view(torch.uint8).view(Bc * Lcap, H * 4))
        vs = float(vc[:, :rows].abs().max().float()) / 448.0
        v8 = torch.empty_like(k8)
        w.wam_quantize_scaled_fp8(vc, vs, v8)
        k8s.append(k8)
        kes.append(ke)
        v8s.append(v8)
        vsc.append(vs)
    torch.cuda.synchronize()
    return k8s, kes, v8s, vsc


class BlockCase:
    """One block over the current chunk of `wl`, given x, e0, ctx and the cache."""

    def __init__(self, wl, layer=0, bias_std=0.0, e0=None, ctx=None):
        self.wl = wl
        B, s = wl.B, wl.seed
        self.W = synth.block_params(wl, layer, bias_std, mod_std=wl.mod_std)
        self.x = synth.normal(s, "x", (B, wl.L, wl.d), 1.0, layer, dtype="f32")
        self.e0 = e0 if e0 is not None else synth.zeros((B, 6, wl.d))
        self.ctx = ctx if ctx is not None else synth.normal(s, "ctx", (B, wl.Lc, wl.d), 1.0, layer)
        self.kc, self.vc = synth.kv_cache(wl, layer, B) if wl.n_cached else (None, None)

    def run_oracle(self, e0=None, ctx=None):
        """fp64 block; e0 / ctx override the seeded ones (float64 arrays)."""
        wl = self.wl
        e0 = self.e0.f64 if e0 is None else e0
        ctx = self.ctx.f64 if ctx is None else ctx
        kp = self.kc.f64 if self.kc is not None else None
        vp = self.vc.f64 if self.vc is not None else None
        return oracle.dit_block(self.x.f64, e0, f64(self.W), wl.H, wl.eps, oracle_positions(wl),
                                np.full(wl.L, wl.n_cached), kp, vp, prev_chunk_ids(wl) if kp is not None else None,
                                ctx=ctx)

    def run_gpu(self, e0_dev=None, ctx_dev=None, fp8=False):
        import torch
        w = lib()
        wl, B = self.wl, self.wl.B
        Wd = {k: dev(v) for k, v in self.W.items()}
        if fp8:
            Wd["fp8"] = w.make_block_fp8(Wd)
        x = dev(self.x)
        kcache, vcache = upload_cache(wl, self.kc, self.vc, B)
        cos, sin = gpu_rope_tables(wl)
        dims = dims_of(wl, 1)
        ws = workspace(w.wam_block_workspace_bytes(dims, B, wl.L, wl.Lc))
        w.wam_dit_block_fwd(dims, w.make_block_weights(Wd), x, dev(self.e0) if e0_dev is None else e0_dev,
                            cos, sin, kcache, vcache, wl.cache_rows, w.cached_chunks(wl.cache_rows, wl.L),
                            ctx=dev(self.ctx) if ctx_dev is None else ctx_dev, ws=ws)
        torch.cuda.synchronize()
        return x, kcache, vcache


# ------------------------------------------------------------------------------ step
class StepCase:
    """A denoising step of `wl` with n_layers seeded blocks (streamed one at a time on the
    oracle side)."""

    def __init__(self, wl, n_layers, bias_std=0.0, flash=False, keep_layers=False):
        """keep_layers: draw each layer once and keep it for both sides (instead of
        drawing it again for the oracle), at the cost of holding every layer in RAM."""
        self.wl, self.n_layers, self.bias_std = wl, n_layers, bias_std
        self.kept = {} if keep_layers else None
        B, s = wl.B, wl.seed
        self.P = synth.model_params(wl, bias_std=bias_std)
        self.z = synth.normal(s, "z_t", (B, wl.latent_ch, wl.F, wl.Hl, wl.Wl), 1.0)
        self.a = synth.normal(s, "a_t", (B, wl.A, wl.act_dim), 1.0)
        self.t = synth.uniform(s, "t", (B,))
        # DreamZero-Flash: the action tokens at their own timestep
        self.t_action = synth.uniform(s, "t_action", (B,)) if flash else None
        self.text = synth.normal(s, "text", (B, wl.Lc, wl.text_dim), 1.0)

    def layer(self, l):
        if self.kept is not None and l in self.kept:
            return self.kept[l]
        W = synth.block_params(self.wl, l, self.bias_std, mod_std=self.wl.mod_std)
        kc, vc = synth.kv_cache(self.wl, l) if self.wl.n_cached else (None, None)
        if self.kept is not None:
            self.kept[l] = (W, kc, vc)
        return W, kc, vc

    def run_oracle(self, depths=None):
        """fp64 velocities; depths: a list of block counts -> the list of velocities after
        each (one pass over the layers)."""
        wl = self.wl

        def layers(l):
            W, kc, vc = self.layer(l)
            return f64(W), (kc.f64 if kc is not None else None), (vc.f64 if vc is not None else None)

        return oracle.dit_step(self.z.f64, self.a.f64, self.t.f64, self.text.f64, f64(self.P), layers,
                               self.n_layers, wl.H, wl.eps, wl.n_cached, oracle_positions(wl),
                               prev_chunk=prev_chunk_ids(wl) if wl.n_cached else None,
                               t_action=self.t_action.f64 if self.t_action is not None else None,
                               depths=depths)

    def upload(self, fp8=False):
        """Device model and inputs (kept on self so the step can be re-run); fp8: the
        blocks carry E4M3 copies of their projections."""
        w = lib()
        wl, B = self.wl, self.wl.B
        self.top = {k: dev(v) for k, v in self.P.items()}
        self.blocks, self.kcs, self.vcs = [], [], []
        for l in range(self.n_layers):
            W, kc, vc = self.layer(l)
            Wd = {k: dev(v) for k, v in W.items()}
            if fp8:
                Wd["fp8"] = w.make_block_fp8(Wd)
            self.blocks.append(Wd)
            k, v = upload_cache(wl, kc, vc, B)
            self.kcs.append(k)
            self.vcs.append(v)
        self.model = w.make_model(dims_of(wl, self.n_layers), self.top, self.blocks)
        self.cos, self.sin = gpu_rope_tables(wl)
        self.dz, self.da, self.dt, self.dtext = dev(self.z), dev(self.a), dev(self.t), dev(self.text)
        self.dta = dev(self.t_action) if self.t_action is not None else None

    def make_fp8_cache(self):
        """E4M3 code caches of the current bf16 caches (fp8_caches), V's scale over the rows
        a step reads and writes (taken after a step with the bf16 cache, a calibration pass)."""
        self.k8s, self.kes, self.v8s, self.vsc = fp8_caches(self.kcs, self.vcs, self.wl.cache_rows + self.wl.L)

    def run_gpu(self, events=None, t_action=None, fp8_cache=False, depth=None):
        """t_action: a device [B] timestep overriding the case's own (None: the case's);
        fp8_cache: run on the E4M3 caches of make_fp8_cache (FP8 self-attention);
        depth: run only the first `depth` blocks (default: all)."""
        import torch
        w = lib()
        wl, B = self.wl, self.wl.B
        if not hasattr(self, "model"):
            self.upload()
        n = self.n_layers if depth is None else depth
        model = self.model if n == self.n_layers else w.make_model(dims_of(wl, n), self.top, self.blocks[:n])
        vv = torch.empty((B, wl.latent_ch, wl.F, wl.Hl, wl.Wl), dtype=torch.float32, device="cuda")
        va = torch.empty((B, wl.A, wl.act_dim), dtype=torch.float32, device="cuda")
        kcs, vcs = (self.k8s, self.v8s) if fp8_cache else (self.kcs, self.vcs)
        io = w.make_step_io(self.dz, self.da, self.dt, self.dtext, kcs[:n], vcs[:n], self.cos, self.sin,
                            wl.cache_rows, w.cached_chunks(wl.cache_rows, wl.L), vv, va, events=events,
                            t_action=t_action if t_action is not None else self.dta,
                            k_exps=self.kes[:n] if fp8_cache else None, v_scales=self.vsc[:n] if fp8_cache else None)
        ws = workspace(w.wam_step_workspace_bytes(model, io))
        w.wam_dit_step_fwd(model, io, ws)
        torch.cuda.synchronize()
        return vv, va


# ------------------------------------------------------------------------------ update pass
class UpdateCase:
    """The cache-update pass over `n_new` clean video-only chunks of `wl` (wl.A must be 0),
    appended after wl.n_cached seeded cached chunks, through n_layers seeded blocks."""

    def __init__(self, wl, n_layers, n_new, t_clean=1.0, bias_std=0.0, spare_rows=64):
        assert wl.A == 0
        self.wl, self.n_layers, self.n_new, self.bias_std = wl, n_layers, n_new, bias_std
        B, s = wl.B, wl.seed
        self.P = synth.model_params(wl, bias_std=bias_std)
        self.z = synth.normal(s, "z_clean", (B, wl.latent_ch, wl.F * n_new, wl.Hl, wl.Wl), 1.0)
        self.a = synth.zeros((B, 0, wl.act_dim), "bf16")
        self.t = synth.Tensor("f32", np.full(B, t_clean, dtype=np.float32))
        self.text = synth.normal(s, "text", (B, wl.Lc, wl.text_dim), 1.0)
        self.L = n_new * wl.L
        self.Lcap = wl.cache_rows + self.L + spare_rows
        self.chunk_ids = np.arange(wl.n_cached, wl.n_cached + n_new)

    def layer(self, l):
        W = synth.block_params(self.wl, l, self.bias_std, mod_std=self.wl.mod_std)
        kc, vc = synth.kv_cache(self.wl, l) if self.wl.n_cached else (None, None)
        return W, kc, vc

    def positions_oracle(self):
        wl = self.wl
        return np.concatenate([oracle.chunk_positions(int(c), wl.F, wl.Hg, wl.Wg, 0) for c in self.chunk_ids])

    def run_oracle(self):
        wl = self.wl

        def layers(l):
            W, kc, vc = self.layer(l)
            return f64(W), (kc.f64 if kc is not None else None), (vc.f64 if vc is not None else None)

        return oracle.dit_update(self.z.f64, self.a.f64, self.t.f64, self.text.f64, f64(self.P), layers,
                                 self.n_layers, wl.H, wl.eps, self.positions_oracle(),
                                 np.repeat(self.chunk_ids, wl.L),
                                 prev_chunk=prev_chunk_ids(wl) if wl.n_cached else None)

    def upload(self):
        import torch
        w = lib()
        wl, B = self.wl, self.wl.B
        self.top = {k: dev(v) for k, v in self.P.items()}
        self.blocks, self.kcs, self.vcs = [], [], []
        for l in range(self.n_layers):
            W, kc, vc = self.layer(l)
            self.blocks.append({k: dev(v) for k, v in W.items()})
            k = torch.zeros((B, self.Lcap, wl.H, wl.Dh), dtype=torch.bfloat16, device="cuda")
            v = torch.zeros_like(k)
            if kc is not None:
                k[:, :wl.cache_rows] = dev(kc)
                v[:, :wl.cache_rows] = dev(vc)
            self.kcs.append(k)
            self.vcs.append(v)
        self.model = w.make_model(dims_of(wl, self.n_layers), self.top, self.blocks)
        self.dz, self.da, self.dt, self.dtext = dev(self.z), dev(self.a), dev(self.t), dev(self.text)

    def run_gpu(self, chunks_at_once=None, fp8_cache=None):
        """Appends the new chunks `chunks_at_once` at a time (default: all in one call).
        Returns the per-layer device caches.  fp8_cache: (k8s, kes, v8s, v_scales) E4M3
        caches to append to instead of the bf16 ones (then those are returned)."""
        import torch
        w = lib()
        wl = self.wl
        if not hasattr(self, "model"):
            self.upload()
        step = chunks_at_once or self.n_new
        cache_len = wl.cache_rows
        for c0 in range(0, self.n_new, step):
            ids = self.chunk_ids[c0:c0 + step]
            pos = np.concatenate([w.wam_chunk_positions(int(c), wl.F, wl.Hg, wl.Wg, 0) for c in ids])
            cos, sin = w.wam_rope_tables(pos, wl.Dh)
            cos, sin = dev(cos), dev(sin)
            z = self.dz[:, :, c0 * wl.F:(c0 + len(ids)) * wl.F].contiguous()
            chunks = w.append_chunks([wl.L] * (wl.n_cached + c0), [wl.L] * len(ids))
            if fp8_cache is None:
                io = w.make_step_io(z, self.da, self.dt, self.dtext, self.kcs, self.vcs, cos, sin, cache_len,
                                    chunks, None, None)
            else:
                k8s, kes, v8s, vsc = fp8_cache
                io = w.make_step_io(z, self.da, self.dt, self.dtext, k8s, v8s, cos, sin, cache_len, chunks, None,
                                    None, k_exps=kes, v_scales=vsc)
            ws = workspace(w.wam_update_workspace_bytes(self.model, io))
            w.wam_dit_update_fwd(self.model, io, ws)
            torch.cuda.synchronize()
            cache_len += len(ids) * wl.L
        return (self.kcs, self.vcs) if fp8_cache is None else (fp8_cache[0], fp8_cache[2])
