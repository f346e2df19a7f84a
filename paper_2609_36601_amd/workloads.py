"""Seeded synthetic logit workloads (student / teacher rows, drafts).

Stand-ins for the paper's Qwen3 student / teacher logits on DAPO-Math
prompts (Sec. 4.1): neither the models nor the data are used.  This module
only draws random numbers; it contains none of the method's arithmetic, so
the HIP path and the CPU oracle can both consume its rows.

Every generator is deterministic given (config, seed, device) and works in
row blocks, so any row range can be regenerated on its own.  Values are drawn
in float32 and rounded once to the stored dtype (round to nearest even).

Configurations (rows = positions):
  tiny    4 seq x 64 pos, V = 4096, float32: s ~ N(0, 2^2);
          t = 0.6 s + 0.8 N(0, 2^2)                                   eps 0.1
  mid     8 seq x 512 pos, V = 32000, bf16: s ~ N(0, 3^2) plus +6 on 320
          (1%) entries per row; t = s + N(0, 1.5^2) (before rounding)  eps 0.05, 0.2
  large   64 seq x 1024 pos, V = 151936, bf16: s ~ N(0, 3^2) / 0.7;
          per sequence rho ~ U(0.3, 0.95); t = rho s + sqrt(1 - rho^2) N(0, 3^2)
                                                                      eps 0.05, 0.2, 0.5
  verify  256 seq x 32 blocks x k = 8, V = 151936, bf16: s as 'large';
          per block rho ~ U(0.2, 0.99); t as 'large'; drafts z_j ~ softmax(s_j)
                                                                      eps 0.2
  stream  32 seq x 8192 pos in chunks of 4096 rows, V = 151936, bf16:
          s ~ N(0, 3^2) / 0.3 plus +12 at one uniform index i; t an independent
          N(0, 3^2) / 0.3 draw plus +12 at i with probability 0.7, else at a
          uniform other index ('shared' variant: t = the student base with the
          spike moved the same way)                                    eps 0.02
"""
import math

import torch

SEED_BASE = 0x5A4B49
VARIANTS = {"": 0, "shared": 1}

CONFIGS = {
    "tiny": dict(index=1, rows=4 * 64, V=4096, dtype=torch.float32, eps=(0.1,), block=256),
    "mid": dict(index=2, rows=8 * 512, V=32000, dtype=torch.bfloat16, eps=(0.05, 0.2), block=512),
    "large": dict(index=3, rows=64 * 1024, V=151936, dtype=torch.bfloat16, eps=(0.05, 0.2, 0.5),
                  block=1024),
    "verify": dict(index=4, rows=256 * 32 * 8, V=151936, dtype=torch.bfloat16, eps=(0.2,), k=8,
                   block=1024),
    "stream": dict(index=5, rows=32 * 8192, V=151936, dtype=torch.bfloat16, eps=(0.02,),
                   block=4096, chunk=4096),
}


def coupling_seed(name):
    return SEED_BASE + CONFIGS[name]["index"]


def _gen(device, *keys):
    g = torch.Generator(device=device)
    h = 1469598103934665603
    for k in keys:
        h = ((h ^ (int(k) & 0xFFFFFFFFFFFF)) * 1099511628211) % (1 << 63)
    g.manual_seed(h)
    return g


def _block_rows(name, seed, device, b, variant=""):
    """Rows of row block b of a configuration as float32 (s, t) before rounding."""
    cfg = CONFIGS[name]
    V, n = cfg["V"], cfg["block"]
    g = _gen(device, seed, cfg["index"], b, VARIANTS[variant])
    if name == "tiny":
        s = 2.0 * torch.randn(n, V, generator=g, device=device)
        t = 0.6 * s + 0.8 * 2.0 * torch.randn(n, V, generator=g, device=device)
    elif name == "mid":
        s = 3.0 * torch.randn(n, V, generator=g, device=device)
        boost = torch.rand(n, V, generator=g, device=device).topk(V // 100, dim=1).indices
        s.scatter_add_(1, boost, torch.full(boost.shape, 6.0, device=device))
        t = s + 1.5 * torch.randn(n, V, generator=g, device=device)
    elif name == "large":
        # one block = one sequence of 1024 positions with its own rho
        rho = 0.3 + 0.65 * torch.rand(1, generator=g, device=device)
        s = 3.0 * torch.randn(n, V, generator=g, device=device) / 0.7
        t = rho * s + torch.sqrt(1 - rho * rho) * 3.0 * torch.randn(n, V, generator=g, device=device)
    elif name == "verify":
        k = cfg["k"]
        rho = 0.2 + 0.79 * torch.rand(n // k, 1, generator=g, device=device)
        rho = rho.repeat_interleave(k, dim=0)
        s = 3.0 * torch.randn(n, V, generator=g, device=device) / 0.7
        t = rho * s + torch.sqrt(1 - rho * rho) * 3.0 * torch.randn(n, V, generator=g, device=device)
    elif name == "stream":
        base_s = 3.0 * torch.randn(n, V, generator=g, device=device) / 0.3
        i = torch.randint(0, V, (n, 1), generator=g, device=device)
        same = torch.rand(n, 1, generator=g, device=device) < 0.7
        other = (i + 1 + torch.randint(0, V - 1, (n, 1), generator=g, device=device)) % V
        j = torch.where(same, i, other)
        base_t = base_s.clone() if variant == "shared" else \
            3.0 * torch.randn(n, V, generator=g, device=device) / 0.3
        s = base_s.scatter_add(1, i, torch.full((n, 1), 12.0, device=device))
        t = base_t.scatter_add(1, j, torch.full((n, 1), 12.0, device=device))
    else:
        raise KeyError(name)
    return s, t


def rows(name, lo, hi, seed=0, device="cpu", variant=""):
    """Stored (student, teacher) logits of rows [lo, hi) of a configuration."""
    cfg = CONFIGS[name]
    nb = cfg["block"]
    out_s, out_t = [], []
    b0, b1 = lo // nb, (hi + nb - 1) // nb
    for b in range(b0, b1):
        s, t = _block_rows(name, seed, device, b, variant)
        a, z = max(lo, b * nb) - b * nb, min(hi, (b + 1) * nb) - b * nb
        out_s.append(s[a:z].to(cfg["dtype"]))
        out_t.append(t[a:z].to(cfg["dtype"]))
        del s, t
    return torch.cat(out_s).contiguous(), torch.cat(out_t).contiguous()


def fill(name, student, teacher, lo=0, seed=0, variant=""):
    """Fill preallocated [n, V] tensors with rows [lo, lo + n) (large configs)."""
    cfg = CONFIGS[name]
    nb = cfg["block"]
    n = student.shape[0]
    r = lo
    while r < lo + n:
        b = r // nb
        hi = min(lo + n, (b + 1) * nb)
        s, t = _block_rows(name, seed, student.device, b, variant)
        a = r - b * nb
        student[r - lo:hi - lo].copy_(s[a:a + hi - r])
        teacher[r - lo:hi - lo].copy_(t[a:a + hi - r])
        del s, t
        r = hi


def drafts(student, seed=0, k=8):
    """Student drafts z_j ~ softmax(s_j) for verify rows (one draw per row)."""
    g = _gen(student.device, seed, 0xD4AF7, student.shape[0])
    out = torch.empty(student.shape[0], dtype=torch.int32, device=student.device)
    step = 2048
    for a in range(0, student.shape[0], step):
        p = torch.softmax(student[a:a + step].float(), dim=-1)
        out[a:a + step] = torch.multinomial(p, 1, generator=g).squeeze(1).to(torch.int32)
    return out


def n_blocks_of(name):
    cfg = CONFIGS[name]
    return math.ceil(cfg["rows"] / cfg["block"])


# ---------------------------------------------------------------------------
# A synthetic autoregressive source: a stand-in for the student and teacher
# networks of a rollout (the paper's engine holds real models; these logits
# depend on the whole prefix through a 64-bit state, so rollouts exercise
# first-rejection commit and rollback).  Pure integer hashing on the host
# (numpy uint64), so every consumer sees the same exact values:
#   state_0(seq)   = mix(seed ^ (seq + 1) * K0)
#   state_{t+1}    = mix(state_t ^ (y_t + 1) * K1)
#   a_v(state)     = mix(state ^ (v + 1) * K2)
#   s_v = ((a_v >> 32) % 33 - 16) / 4            (student, in [-4, 4])
#   t_v = s_v / 2 + ((a_v & 0xffffffff) % 17 - 8) / 4   (teacher, multiples of 1/8)
# mix is the SplitMix64 output function (Steele, Lea, Flood, OOPSLA 2014).
# All values are exact in bf16, f32 and f64.
# ---------------------------------------------------------------------------
_M64 = (1 << 64) - 1
_K0, _K1, _K2 = 0x9E3779B97F4A7C15, 0xD6E8FEB86659FD93, 0xA0761D6478BD642F


def _mix(x):
    import numpy as np
    x = np.asarray(x, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = x + np.uint64(0x9E3779B97F4A7C15)
        z = (z ^ (z >> np.uint64(30))) * np.uint64(0xBF58476D1CE4E5B9)
        z = (z ^ (z >> np.uint64(27))) * np.uint64(0x94D049BB133111EB)
        return z ^ (z >> np.uint64(31))


class SyntheticAR:
    """Prefix-hash student/teacher logits over V tokens (see above)."""

    def __init__(self, V, seed=0):
        self.V = int(V)
        self.seed = int(seed) & _M64

    def initial(self, seq_ids):
        import numpy as np
        seq = np.asarray(seq_ids, dtype=np.uint64)
        with np.errstate(over="ignore"):
            return _mix(np.uint64(self.seed) ^ ((seq + np.uint64(1)) * np.uint64(_K0)))

    def advance(self, states, tokens):
        import numpy as np
        tok = np.asarray(tokens, dtype=np.int64).astype(np.uint64)
        with np.errstate(over="ignore"):
            return _mix(np.asarray(states, dtype=np.uint64) ^ ((tok + np.uint64(1)) * np.uint64(_K1)))

    def logits(self, states):
        """(s, t) as float32 arrays [len(states), V] (exact values)."""
        import numpy as np
        st = np.asarray(states, dtype=np.uint64)[:, None]
        v = np.arange(self.V, dtype=np.uint64)[None, :]
        with np.errstate(over="ignore"):
            a = _mix(st ^ ((v + np.uint64(1)) * np.uint64(_K2)))
        hi = (a >> np.uint64(32)).astype(np.int64)
        lo = (a & np.uint64(0xFFFFFFFF)).astype(np.int64)
        s = ((hi % 33) - 16).astype(np.float32) / 4.0
        t = s / 2.0 + ((lo % 17) - 8).astype(np.float32) / 4.0
        return s, t


def _i64(c):
    """A uint64 constant as the int64 with the same bits."""
    return c - (1 << 64) if c >= (1 << 63) else c


def _mix_t(x):
    """SplitMix64 output function on int64 tensors (two's-complement wrap)."""
    def srl(v, k):
        return (v >> k) & ((1 << (64 - k)) - 1)
    z = x + _i64(0x9E3779B97F4A7C15)
    z = (z ^ srl(z, 30)) * _i64(0xBF58476D1CE4E5B9)
    z = (z ^ srl(z, 27)) * _i64(0x94D049BB133111EB)
    return z ^ srl(z, 31)


class SyntheticARTorch:
    """SyntheticAR on int64 torch tensors (any device): same states and logits."""

    def __init__(self, V, seed=0, device="cpu"):
        self.V = int(V)
        self.seed = _i64(int(seed) & _M64)
        self.device = device

    def initial(self, seq_ids):
        import torch
        seq = torch.as_tensor(seq_ids, dtype=torch.int64, device=self.device)
        return _mix_t(self.seed ^ ((seq + 1) * _i64(_K0)))

    def advance(self, states, tokens):
        import torch
        tok = tokens.to(torch.int64)
        return _mix_t(states ^ ((tok + 1) * _i64(_K1)))

    def logits_into(self, states, s_out=None, t_out=None):
        """Writes s and/or t for `states` [n] into [n, V] views (any float dtype)."""
        import torch
        v = torch.arange(self.V, dtype=torch.int64, device=states.device)
        a = _mix_t(states[:, None] ^ ((v[None, :] + 1) * _i64(_K2)))
        hi = (a >> 32) & 0xFFFFFFFF
        s = ((hi % 33) - 16).to(torch.float32) / 4.0
        if s_out is not None:
            s_out.copy_(s)
        if t_out is not None:
            lo = a & 0xFFFFFFFF
            t_out.copy_(s / 2.0 + ((lo % 17) - 8).to(torch.float32) / 4.0)
