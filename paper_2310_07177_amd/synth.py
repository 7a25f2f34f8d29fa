"""Seeded synthetic inputs shaped like the paper's draft/target logit pairs.

This module is shared by the tests, the benchmark and the smoke check, and
feeds identical bits to the HIP library and to the CPU oracle.  It holds none
of the verification or distillation arithmetic: it draws logits, proposal
tokens, uniforms, masks and proposal lengths, and nothing else.

Conventions:
  * logits are drawn as float32 normals and stored either as float32 or as
    bf16 bit patterns (uint16) rounded to nearest-even;
  * uniforms are k * 2^-24 for integer k in [0, 2^24), so they lie in [0, 1)
    and are exact in float32;
  * proposal tokens y_i ~ softmax(d_i / T) are drawn with the Gumbel-max trick
    on the stored (rounded) draft logits, so they follow the distribution the
    kernels will see; T == 0 takes the draft argmax;
  * seeds: uniforms 0, logits 1, proposal draws 2, masks/peaks/lengths 3
    (offset by the caller's base seed).

The workloads stand in for the paper's (Section 5: Vicuna/LLaMA vocabularies
of about 32k and the T5 vocabulary); the paper's datasets and weights are not
used.
"""
from __future__ import annotations

import numpy as np

SEED_UNIFORM, SEED_LOGITS, SEED_TOKENS, SEED_AUX = 0, 1, 2, 3


def rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def uniforms(g: np.random.Generator, shape) -> np.ndarray:
    """float32 uniforms k * 2^-24, k uniform in [0, 2^24): in [0, 1), never 1."""
    return (g.integers(0, 1 << 24, size=shape, dtype=np.int64).astype(np.float32)
            * np.float32(2.0 ** -24))


def to_bf16(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest even."""
    x = np.ascontiguousarray(x, np.float32)
    b = x.view(np.uint32).astype(np.uint64)
    b = (b + 0x7FFF + ((b >> 16) & 1)) >> 16
    out = b.astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        out[nan] = 0x7FC0
    return out


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    b = np.ascontiguousarray(bits, np.uint16).astype(np.uint32) << 16
    return b.view(np.float32)


def store(x: np.ndarray, dtype: str) -> np.ndarray:
    """Store float32 logits in the requested format ('f32' or 'bf16')."""
    if dtype == "f32":
        return np.ascontiguousarray(x, np.float32)
    if dtype == "bf16":
        return to_bf16(x)
    raise ValueError(dtype)


def as_f32(stored: np.ndarray) -> np.ndarray:
    return bf16_to_f32(stored) if stored.dtype == np.uint16 else stored


def gumbel_max_tokens(g: np.random.Generator, draft_stored: np.ndarray,
                      T: float, chunk_rows: int = 256) -> np.ndarray:
    """y[..., i] ~ softmax(draft[..., i, :] / T) by the Gumbel-max trick
    (argmax of logits/T plus i.i.d. Gumbel noise); T == 0 gives the argmax."""
    lead = draft_stored.shape[:-1]
    V = draft_stored.shape[-1]
    rows = draft_stored.reshape(-1, V)
    out = np.empty(rows.shape[0], np.int32)
    for r0 in range(0, rows.shape[0], chunk_rows):
        z = as_f32(rows[r0:r0 + chunk_rows]).astype(np.float64)
        if T > 0:
            u = g.random(z.shape)
            u = np.clip(u, 1e-300, 1.0)
            z = z / T - np.log(-np.log(u))
        out[r0:r0 + chunk_rows] = np.argmax(z, axis=-1)
    return out.reshape(lead)


def normals(g: np.random.Generator, shape, std: float) -> np.ndarray:
    return g.standard_normal(size=shape, dtype=np.float32) * np.float32(std)


# --------------------------------------------------------------------------
# Workloads.  Each returns a dict of numpy arrays plus the scalar settings.
# --------------------------------------------------------------------------

def verify_inputs(B, K, V, dtype="bf16", T=1.0, seed=0, target_std=2.0,
                  draft_scale=1.0, draft_noise=1.0, peaks=0, peak_boost=8.0,
                  ragged=False):
    """Generic verification inputs: target ~ N(0, target_std^2) (+ optional
    per-row peaks), draft = draft_scale * target + N(0, draft_noise^2)."""
    gl = rng(seed * 16 + SEED_LOGITS)
    ga = rng(seed * 16 + SEED_AUX)
    t = normals(gl, (B, K + 1, V), target_std)
    if peaks:
        for b in range(B):
            for i in range(K + 1):
                ids = ga.choice(V, size=min(peaks, V), replace=False)
                t[b, i, ids] += np.float32(peak_boost)
    d = np.float32(draft_scale) * t[:, :K, :] + normals(gl, (B, K, V), draft_noise)
    target = store(t, dtype)
    draft = store(d, dtype)
    tokens = gumbel_max_tokens(rng(seed * 16 + SEED_TOKENS), draft, T)
    gu = rng(seed * 16 + SEED_UNIFORM)
    u_acc = uniforms(gu, (B, K))
    u_res = uniforms(gu, (B,))
    draft_len = ga.integers(1, K + 1, size=B).astype(np.int32) if ragged else None
    return dict(target=target, draft=draft, tokens=tokens, u_accept=u_acc,
                u_resample=u_res, draft_len=draft_len, T=float(T), B=B, K=K, V=V,
                dtype=dtype)


def config_tiny(seed=0):
    """B=1, k=4, V=1000 fp32; target ~ N(0, 2^2), draft = target + N(0, 1);
    T=1; forward KL over all k positions."""
    x = verify_inputs(1, 4, 1000, "f32", T=1.0, seed=seed, target_std=2.0,
                      draft_noise=1.0)
    x.update(kind="fkl", beta=0.5, tau=1.0, mask=np.ones((1, 4), np.uint8))
    return x


def config_llama_vocab(sigma=1.0, seed=0):
    """B=8, k=5, V=32000 bf16; target ~ N(0, 3^2) with 20 random peak tokens
    per row boosted by +8; draft = target + N(0, sigma^2); T=1; forward KL on
    the rejected positions."""
    x = verify_inputs(8, 5, 32000, "bf16", T=1.0, seed=seed, target_std=3.0,
                      draft_noise=sigma, peaks=20, peak_boost=8.0)
    x.update(kind="fkl", beta=0.5, tau=1.0, mask=None)
    return x


def config_t5_vocab(seed=0, greedy=False, B=64, K=8):
    """B=64, k=8, V=32128 bf16; target ~ N(0, 2.5^2), draft = 0.7 target +
    N(0, 1.5^2); T=0.7 (or greedy, T=0); distillation at tau=0.7 over all
    positions with the first K target rows as teacher."""
    T = 0.0 if greedy else 0.7
    x = verify_inputs(B, K, 32128, "bf16", T=T, seed=seed, target_std=2.5,
                      draft_scale=0.7, draft_noise=1.5)
    x.update(tau=0.7, beta=0.5, mask=np.ones((B, K), np.uint8))
    return x


def zipf_bias(V, seed=0, s=1.1):
    """b_j = -s * ln(rank_j) for one seeded permutation of ranks 1..V, so that
    softmax(b) is a Zipf(s) law over the vocabulary."""
    ranks = rng(seed * 16 + SEED_AUX).permutation(V).astype(np.float64) + 1.0
    return (-s * np.log(ranks)).astype(np.float32)


def config_distill_buffer(N=16384, V=32000, seed=0, mask_p=0.4, chunk=1024):
    """N buffered positions (B=N, K=1), V=32000 bf16: teacher ~ N(0, 3^2) plus
    a Zipf(1.1)-ranked bias; student = teacher + N(0, 1); JSD(beta=0.5),
    tau=1, mean loss over a Bernoulli(0.4) mask, full bf16 gradient."""
    gl = rng(seed * 16 + SEED_LOGITS)
    bias = zipf_bias(V, seed)
    teacher = np.empty((N, 1, V), np.uint16)
    student = np.empty((N, 1, V), np.uint16)
    for r0 in range(0, N, chunk):
        n = min(chunk, N - r0)
        t = normals(gl, (n, V), 3.0) + bias
        s = t + normals(gl, (n, V), 1.0)
        teacher[r0:r0 + n, 0] = to_bf16(t)
        student[r0:r0 + n, 0] = to_bf16(s)
    mask = (rng(seed * 16 + SEED_AUX + 1).random((N, 1)) < mask_p).astype(np.uint8)
    return dict(teacher=teacher, student=student, mask=mask, kind="jsd", beta=0.5,
                tau=1.0, B=N, K=1, V=V, dtype="bf16")


def sample_inputs(N, V, dtype="bf16", seed=0, p_std=3.0, q_noise=1.0, zipf=False):
    """Rows for token sampling: p ~ N(0, p_std^2) (plus a Zipf(1.1)-ranked
    bias when zipf), q = p + N(0, q_noise^2), and one uniform per row."""
    gl = rng(seed * 16 + SEED_LOGITS)
    t = normals(gl, (N, V), p_std)
    if zipf:
        t = t + zipf_bias(V, seed)
    d = t + normals(gl, (N, V), q_noise)
    u = uniforms(rng(seed * 16 + SEED_UNIFORM), N)
    return dict(p=store(t, dtype), q=store(d, dtype), u=u, N=N, V=V, dtype=dtype)


def config_large_vocab(seed=0, B=256, K=8, V=128256):
    """B=256 sequences with ragged proposal lengths k_b ~ U{1..8}, V=128256
    bf16; target ~ N(0, 3^2), draft = target + N(0, 1); T=0.8; forward KL at
    tau=0.8 on the rejected positions."""
    x = verify_inputs(B, K, V, "bf16", T=0.8, seed=seed, target_std=3.0,
                      draft_noise=1.0, ragged=True)
    x.update(kind="fkl", beta=0.5, tau=0.8, mask=None)
    return x


def config_large_vocab_device(seed=0, B=256, K=8, V=128256, device="cuda"):
    """The large-vocabulary workload at its full size, drawn on the GPU with
    torch's seeded generator (the host generator takes minutes at 0.6 G
    logits): target ~ N(0, 3^2), draft = target + N(0, 1), both float32
    normals rounded once to bf16; k_b ~ U{1..8}; proposals by Gumbel-max on
    the stored draft logits at T = 0.8; float32 uniforms in [0, 1).  Returns
    device tensors (target and draft bf16, tokens and draft_len int32,
    uniforms float32) plus the scalar settings; slices of them, copied to the
    host, are the oracle's inputs."""
    import torch
    T = 0.8
    g = torch.Generator(device=device)
    g.manual_seed(seed * 16 + SEED_LOGITS)
    t = torch.randn(B, K + 1, V, generator=g, device=device) * 3.0
    d = (t[:, :K] + torch.randn(B, K, V, generator=g, device=device)).to(torch.bfloat16)
    t = t.to(torch.bfloat16)
    gt = torch.Generator(device=device)
    gt.manual_seed(seed * 16 + SEED_TOKENS)
    tokens = torch.empty(B, K, dtype=torch.int32, device=device)
    for b0 in range(0, B, 32):  # bounded temporaries
        u = torch.rand(min(32, B - b0), K, V, generator=gt, device=device).clamp_min_(1e-30)
        gum = -torch.log(-torch.log(u))
        tokens[b0:b0 + 32] = torch.argmax(d[b0:b0 + 32].float() / T + gum, dim=-1).to(torch.int32)
    gu = torch.Generator(device=device)
    gu.manual_seed(seed * 16 + SEED_UNIFORM)
    u_acc = torch.rand(B, K, generator=gu, device=device)
    u_res = torch.rand(B, generator=gu, device=device)
    ga = torch.Generator(device=device)
    ga.manual_seed(seed * 16 + SEED_AUX)
    draft_len = torch.randint(1, K + 1, (B,), generator=ga, device=device, dtype=torch.int32)
    return dict(target=t, draft=d, tokens=tokens, u_accept=u_acc, u_resample=u_res, draft_len=draft_len,
                T=T, B=B, K=K, V=V, dtype="bf16", kind="fkl", beta=0.5, tau=T)


def to_host_sample(x, idx):
    """Host copies (numpy, bf16 as uint16 bit patterns) of the sequences idx
    of a device workload, in the layout the oracle takes."""
    import torch
    ii = torch.as_tensor(np.asarray(idx), device=x["target"].device)

    def h(t):
        s = t.index_select(0, ii).contiguous().cpu()
        if s.dtype == torch.bfloat16:
            return s.view(torch.int16).numpy().view(np.uint16)
        return s.numpy()
    return dict(target=h(x["target"]), draft=h(x["draft"]), tokens=h(x["tokens"]), u_accept=h(x["u_accept"]),
                u_resample=h(x["u_resample"]), draft_len=h(x["draft_len"]), T=x["T"], B=len(idx), K=x["K"],
                V=x["V"], dtype=x["dtype"])


def tree_parents(branching, max_nodes=64) -> np.ndarray:
    """Parent array of a candidate tree built level by level: every node of
    level l gets branching[l] children, nodes numbered breadth-first (so each
    parent precedes its children), truncated to max_nodes.  [-1] is the root."""
    parent = [-1]
    level = [0]
    for nb in branching:
        nxt = []
        for v in level:
            for _ in range(nb):
                if len(parent) >= max_nodes:
                    break
                nxt.append(len(parent))
                parent.append(v)
        level = nxt
    return np.array(parent, np.int32)


def random_tree_parents(g: np.random.Generator, N: int) -> np.ndarray:
    """A random tree on N nodes: node n's parent is uniform over 0..n-1."""
    par = np.full(N, -1, np.int32)
    for n in range(1, N):
        par[n] = g.integers(0, n)
    return par


def tree_inputs(B, parent, V, dtype="bf16", T=1.0, seed=0, target_std=2.0, draft_scale=1.0, draft_noise=1.0):
    """Tree verification inputs: per sequence the tree `parent` ([N] shared,
    or [B, N]); target rows ~ N(0, target_std^2), draft rows = draft_scale *
    target + N(0, draft_noise^2); node n's token ~ softmax(draft[parent[n]] /
    T) by Gumbel-max (the argmax at T == 0); uniforms on the 2^-24 grid."""
    par = np.asarray(parent, np.int32)
    if par.ndim == 1:
        par = np.tile(par, (B, 1))
    N = par.shape[1]
    gl = rng(seed * 16 + SEED_LOGITS)
    t = normals(gl, (B, N, V), target_std)
    d = (np.float32(draft_scale) * t + normals(gl, (B, N, V), draft_noise)).astype(np.float32)
    target, draft = store(t, dtype), store(d, dtype)
    # proposals: node n's token is an independent draw from its parent's
    # draft row (siblings are i.i.d. candidates)
    bi = np.repeat(np.arange(B), N - 1)
    pi = np.maximum(par[:, 1:], 0).reshape(-1)
    tokens = np.zeros((B, N), np.int32)
    tokens[:, 1:] = gumbel_max_tokens(rng(seed * 16 + SEED_TOKENS), draft[bi, pi], T).reshape(B, N - 1)
    gu = rng(seed * 16 + SEED_UNIFORM)
    return dict(target=target, draft=draft, parent=par, tokens=tokens, u_accept=uniforms(gu, (B, N)),
                u_resample=uniforms(gu, B), T=T, B=B, N=N, V=V)


def config_medusa_tree(seed=0, B=16, V=32000, branching=(4, 3, 2, 1), max_nodes=64):
    """A Medusa-style candidate tree per sequence (Section 5, OSD + Medusa on
    a Vicuna-7B-size vocabulary): branching 4, 3, 2, 1 by level, 64 nodes;
    target ~ N(0, 3^2), draft = target + N(0, 1^2), T = 1."""
    return tree_inputs(B, tree_parents(branching, max_nodes), V, "bf16", T=1.0, seed=seed, target_std=3.0,
                       draft_noise=1.0)
