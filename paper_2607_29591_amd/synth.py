"""Seeded synthetic inputs for the ResKV workloads.

This module only draws random numbers and lays them out; it holds none of
the method's arithmetic. Both the GPU path and the fp64 checker consume what
it produces, so they read identical bits.

Recipe (LLM-shaped key/value statistics):
  * keys   ~ N(0, 1), plus a per-channel bias ~ N(0, sigma=3) on 4 channels
    that are fixed per (layer, KV head);
  * a set of "heavy" positions (uniform over the context, distinct) whose keys
    are scaled by 3 after the bias is added;
  * values ~ N(0, 1);
  * every query (observation window and decode) of a query head is
    0.7 * mean(4 distinct random heavy keys of its KV head) + 0.3 * N(0, 1);
  * bf16 workloads round every drawn value once, to nearest-even.

The five workloads mirror a single-layer fp32 toy, a Llama-3.1-8B-shaped layer
(32 q / 8 KV heads, head_dim 128), a batched 32-layer decode, a long-context
construction-heavy case and a ragged 28 q / 4 KV head (GQA 7) batch.
"""

from dataclasses import dataclass, field

import numpy as np

SEED = 42


@dataclass
class Workload:
    name: str
    batch: int
    layers: int
    hq: int
    hkv: int
    d: int
    dtype: str                 # "f32" or "bf16"
    ctx: list                  # per-sequence context length
    n_heavy: list              # per-sequence heavy-token count
    window: int                # observation window w (= protected recent window)
    budget: list               # per-sequence budget b
    res: np.ndarray            # [layers, batch, hkv] residual count r
    steps: int                 # decode steps
    appends: bool              # decode appends the new token's K/V each step
    tau: object = 0.25         # scalar, or "normal" for per-query N(0, 0.5)
    alpha: float = 12.0
    g_min: float = 0.0
    beta: float = 1.0
    lloyd_iters: int = 4
    extra: dict = field(default_factory=dict)

    @property
    def group(self):
        return self.hq // self.hkv

    @property
    def max_ctx(self):
        return int(max(self.ctx))

    @property
    def slot_cap(self):
        """Slots per (sequence, KV head): the budget plus room for appends."""
        return int(max(self.budget)) + (self.steps if self.appends else 0)

    @property
    def res_cap(self):
        return int(max(1, self.res.max()))


def workload(i, seed=SEED):
    """The i-th workload (0..4); random per-head splits are seeded."""
    rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 1000 + i])))
    if i == 0:
        return Workload("toy-fp32-gqa4-d64-ctx1k", 1, 1, 8, 2, 64, "f32", [1024], [8], 16,
                        [128], np.full((1, 1, 2), 32), 8, False)
    if i == 1:
        res = rng.choice([0, 16, 32, 64, 128], size=(1, 1, 8))
        return Workload("llama8b-layer-ctx32k-b512", 1, 1, 32, 8, 128, "bf16", [32768], [64], 32,
                        [512], res, 128, False)
    if i == 2:
        res = rng.choice([0, 64, 128, 256, 512], size=(32, 1, 8))
        res = np.repeat(res, 32, axis=1)
        return Workload("llama8b-32L-b32-ctx32k-b2048-decode", 32, 32, 32, 8, 128, "bf16",
                        [32768] * 32, [64] * 32, 32, [2048] * 32, res, 256, True, tau="normal")
    if i == 3:
        return Workload("llama8b-8L-b4-ctx128k-b1024-build", 4, 8, 32, 8, 128, "bf16",
                        [131072] * 4, [1311] * 4, 64, [1024] * 4, np.full((8, 4, 8), 256), 64, True)
    if i == 4:
        ctx = rng.integers(4096, 65536, size=64, endpoint=True)
        budget = rng.choice([256, 512, 1024], size=64)
        frac = rng.uniform(0.0, 0.5, size=(28, 1, 4))
        res = 16 * np.floor(frac * budget[None, :, None] / 16 + 0.5).astype(np.int64)
        return Workload("qwen7b-28L-b64-ragged-ctx4k-64k", 64, 28, 28, 4, 128, "bf16",
                        [int(c) for c in ctx], [int(c) // 512 for c in ctx], 32,
                        [int(b) for b in budget], res, 128, True)
    raise ValueError(i)


def tiny_workload(s=40, d=8, hq=4, hkv=2, budget=16, res=4, window=4, n_heavy=3,
                  dtype="f32", batch=1, steps=2):
    """A small workload for unit tests (sizes chosen by the caller)."""
    return Workload("tiny", batch, 1, hq, hkv, d, dtype, [s] * batch, [n_heavy] * batch, window,
                    [budget] * batch, np.full((1, batch, hkv), res), steps, False)


# --------------------------------------------------------------------------
# numpy generator (host): small and medium workloads, and checker samples
# --------------------------------------------------------------------------

def _bf16_bits_round(x):
    """float32 -> nearest-even bf16 value, returned as float32."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32).astype(np.uint64)
    u = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return (u.astype(np.uint32) << 16).view(np.float32)


def _store(x, dtype):
    x = np.asarray(x, dtype=np.float32)
    return _bf16_bits_round(x) if dtype == "bf16" else x


def _rng(seed, *key):
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, *key])))


def _head_keys(rng, s, d, n_heavy):
    ch = rng.choice(d, size=4, replace=False)
    bias = np.zeros(d, np.float32)
    bias[ch] = rng.normal(0.0, 3.0, size=4)
    K = rng.standard_normal((s, d), dtype=np.float32) + bias
    heavy = np.sort(rng.choice(s, size=max(1, min(n_heavy, s)), replace=False))
    K[heavy] *= 3.0
    return K, heavy, bias


def _queries(rng, K, heavy, n, d):
    pick = np.stack([rng.choice(heavy, size=min(4, heavy.size), replace=False) for _ in range(n)])
    return (0.7 * K[pick].mean(axis=1) + 0.3 * rng.standard_normal((n, d), dtype=np.float32))


def gen_layer(wl, layer=0, seed=SEED, n_decode=None):
    """Host tensors for one layer of workload `wl`.

    Returns a dict of float32 numpy arrays (already rounded to the storage
    dtype): K, V [B, Hkv, S, d] (rows past a sequence's length are zero),
    q_obs [B, Hq, w, d], q_dec [steps, B, Hq, d], k_new, v_new
    [steps, B, Hkv, d] (appended tokens), tau [steps, B, Hq], plus int arrays
    seq_len [B], budget [B], res [B, Hkv].
    """
    B, Hkv, G, d, w = wl.batch, wl.hkv, wl.group, wl.d, wl.window
    S = wl.max_ctx
    steps = wl.steps if n_decode is None else n_decode
    K = np.zeros((B, Hkv, S, d), np.float32)
    V = np.zeros((B, Hkv, S, d), np.float32)
    q_obs = np.zeros((B, wl.hq, w, d), np.float32)
    q_dec = np.zeros((steps, B, wl.hq, d), np.float32)
    k_new = np.zeros((steps, B, Hkv, d), np.float32)
    v_new = np.zeros((steps, B, Hkv, d), np.float32)
    for b in range(B):
        s = wl.ctx[b]
        for h in range(Hkv):
            rng = _rng(seed, layer, b, h)
            Kh, heavy, bias = _head_keys(rng, s, d, wl.n_heavy[b])
            Kh = _store(Kh, wl.dtype)
            K[b, h, :s] = Kh
            V[b, h, :s] = _store(rng.standard_normal((s, d), dtype=np.float32), wl.dtype)
            for g in range(G):
                q_obs[b, h * G + g] = _store(_queries(rng, Kh, heavy, w, d), wl.dtype)
                q_dec[:, b, h * G + g] = _store(_queries(rng, Kh, heavy, steps, d), wl.dtype)
            k_new[:, b, h] = _store(rng.standard_normal((steps, d), dtype=np.float32) + bias, wl.dtype)
            v_new[:, b, h] = _store(rng.standard_normal((steps, d), dtype=np.float32), wl.dtype)
    trng = _rng(seed, layer, 7777)
    if wl.tau == "normal":
        tau = trng.normal(0.0, 0.5, size=(steps, B, wl.hq)).astype(np.float32)
    else:
        tau = np.full((steps, B, wl.hq), wl.tau, np.float32)
    return dict(K=K, V=V, q_obs=q_obs, q_dec=q_dec, k_new=k_new, v_new=v_new, tau=tau,
                seq_len=np.asarray(wl.ctx, np.int32), budget=np.asarray(wl.budget, np.int32),
                res=np.asarray(wl.res[layer], np.int32))


# --------------------------------------------------------------------------
# torch generator (device): full-size workloads generated in HBM
# --------------------------------------------------------------------------

def gen_layer_device(wl, layer, device, seed=SEED, n_decode=None, out=None):
    """Device tensors for one layer, drawn with a seeded device generator.

    Same recipe and layout as gen_layer, stored in the workload dtype
    (torch.bfloat16 or torch.float32), vectorised over the KV heads of each
    sequence. `out` may hold preallocated K, V (rows past a sequence's length
    are left as they are: nothing reads them).
    """
    import torch
    tdt = torch.bfloat16 if wl.dtype == "bf16" else torch.float32
    B, Hkv, G, d, w = wl.batch, wl.hkv, wl.group, wl.d, wl.window
    S = wl.max_ctx
    steps = wl.steps if n_decode is None else n_decode
    gen = torch.Generator(device=device)
    gen.manual_seed(int(np.random.SeedSequence([seed, layer, 31337]).generate_state(1)[0]))
    f32 = dict(dtype=torch.float32, device=device, generator=gen)
    out = {} if out is None else out
    K = out.get("K")
    V = out.get("V")
    if K is None:
        K = torch.empty((B, Hkv, S, d), dtype=tdt, device=device)
        V = torch.empty((B, Hkv, S, d), dtype=tdt, device=device)
    q_obs = torch.empty((B, wl.hq, w, d), dtype=tdt, device=device)
    q_dec = torch.empty((steps, B, wl.hq, d), dtype=tdt, device=device)
    k_new = torch.empty((steps, B, Hkv, d), dtype=tdt, device=device)
    v_new = torch.empty((steps, B, Hkv, d), dtype=tdt, device=device)

    def queries(hk, n):
        # [Hkv, G, n, d]: 0.7 * mean of 4 distinct heavy keys + 0.3 * N(0, 1)
        nh = hk.shape[1]
        pick = torch.rand((Hkv, G, n, nh), **f32).argsort(dim=-1)[..., :min(4, nh)]
        src = hk[:, None, None].expand(Hkv, G, n, nh, d)
        sel = torch.gather(src, 3, pick[..., None].expand(*pick.shape, d))
        return 0.7 * sel.mean(dim=3) + 0.3 * torch.randn((Hkv, G, n, d), **f32)

    for b in range(B):
        s = int(wl.ctx[b])
        nh = max(1, min(int(wl.n_heavy[b]), s))
        ch = torch.rand((Hkv, d), **f32).argsort(dim=-1)[:, :4]
        bias = torch.zeros((Hkv, d), dtype=torch.float32, device=device)
        bias.scatter_(1, ch, 3.0 * torch.randn((Hkv, 4), **f32))
        kh = torch.randn((Hkv, s, d), **f32) + bias[:, None, :]
        heavy = torch.rand((Hkv, s), **f32).argsort(dim=-1)[:, :nh]
        idx = heavy[:, :, None].expand(Hkv, nh, d)
        kh.scatter_(1, idx, kh.gather(1, idx) * 3.0)
        khs = kh.to(tdt)
        del kh
        K[b, :, :s] = khs
        V[b, :, :s] = torch.randn((Hkv, s, d), **f32).to(tdt)
        hk = khs.gather(1, idx).float()
        q_obs[b] = queries(hk, w).reshape(Hkv * G, w, d).to(tdt)
        q_dec[:, b] = queries(hk, steps).permute(2, 0, 1, 3).reshape(steps, Hkv * G, d).to(tdt)
        k_new[:, b] = (torch.randn((steps, Hkv, d), **f32) + bias).to(tdt)
        v_new[:, b] = torch.randn((steps, Hkv, d), **f32).to(tdt)
    if wl.tau == "normal":
        tau = 0.5 * torch.randn((steps, B, wl.hq), **f32)
    else:
        tau = torch.full((steps, B, wl.hq), float(wl.tau), dtype=torch.float32, device=device)
    return dict(K=K, V=V, q_obs=q_obs, q_dec=q_dec, k_new=k_new, v_new=v_new, tau=tau,
                seq_len=np.asarray(wl.ctx, np.int32), budget=np.asarray(wl.budget, np.int32),
                res=np.asarray(wl.res[layer], np.int32))
