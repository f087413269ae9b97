"""FeatFix oracle: plain fp64 NumPy statement of the cached DiT denoising loop.

TEST INFRASTRUCTURE ONLY (see the package docstring).  No blocking, fusion or
reordering beyond the definitions cited on each function.

Paper passages followed (section / equation of the FeatFix paper):
  * Sec. 3.1, Eq. 1   -- exact block output h_f = B_l(u; t, c).
  * Sec. 3.1, Eq. 2   -- order-K Taylor draft from finite differences estimated at
                         exact refreshes; order 0 is plain reuse of the refreshed feature.
  * Sec. 3.1, Eq. 3   -- same-input pair (draft and exact from one incoming state).
  * Sec. 3.1, Eq. 4   -- normalised relative-L1 discrepancy with eps > 0 (audit only).
  * Sec. 3.3, Eq. 5   -- forwarding rule: exact output at sites, draft elsewhere.
  * Sec. 3.3, "Matched-compute controls and accounting" -- Verify forwards the draft,
    Exact-only forwards the exact output without the draft/discrepancy paths; full
    refreshes, paid checks and forwarded corrections are counted separately.

Readings where the paper is silent (block internals, residual caching, the
finite-difference recursion, refresh rule, sampler, conditioning, precision) are the
ones listed in the design notes; each is restated where it is used below.
"""
from __future__ import annotations

import math
import numpy as np

DIT, MMDIT_DOUBLE, MMDIT_SINGLE = 0, 1, 2
F32, BF16 = 0, 1
VANILLA, DRAFT, VERIFY, FEATFIX, EXACT_ONLY = 0, 1, 2, 3, 4
TOKENS_PARTIAL, CHANNELS_PARTIAL, RECOMPUTE = 5, 6, 7   # the matched-compute arms of Sec. 3.3
PAID_MODES = (VERIFY, FEATFIX, EXACT_ONLY, TOKENS_PARTIAL, CHANNELS_PARTIAL, RECOMPUTE)
FORWARDING_MODES = (FEATFIX, EXACT_ONLY, TOKENS_PARTIAL, CHANNELS_PARTIAL, RECOMPUTE)
RESIDUAL, OUTPUT = 0, 1
REFRESH_STEP, CACHED_STEP = 0, 1
EXACT, DRAFT_ACT, SITE, RECOMPUTE_ACT = 0, 1, 2, 3
TEMB_DIM = 256

__all__ = [
    "DIT", "MMDIT_DOUBLE", "MMDIT_SINGLE", "F32", "BF16", "VANILLA", "DRAFT", "VERIFY",
    "FEATFIX", "EXACT_ONLY", "TOKENS_PARTIAL", "CHANNELS_PARTIAL", "RECOMPUTE", "PAID_MODES",
    "FORWARDING_MODES", "RESIDUAL", "OUTPUT", "REFRESH_STEP", "CACHED_STEP", "EXACT",
    "DRAFT_ACT", "SITE", "RECOMPUTE_ACT", "forward_partial", "round_bf16", "silu", "gelu_tanh", "layer_norm", "rms_norm",
    "softmax", "attention", "timestep_embedding", "conditioning", "patchify", "unpatchify",
    "dit_block", "double_block", "single_block", "block", "rope", "rope_positions", "final_layer", "make_plan",
    "TaylorCache", "rel_l1", "run", "max_rel_err", "block_flops",
]


# ----------------------------------------------------------------------------- precision

def round_bf16(x):
    """Round to the nearest bfloat16 value, ties to even, straight from fp64.

    bf16 has 8 significant bits and fp32's exponent range: the spacing of bf16 values
    around x is 2**(e-8) for x = m * 2**e with m in [0.5, 1) (normal range e >= -125),
    and 2**-133 below it (subnormals).  Beyond the largest finite bf16 the value is inf.
    """
    x = np.asarray(x, dtype=np.float64)
    _, e = np.frexp(x)
    spacing = np.ldexp(1.0, np.maximum(e, -125) - 8)
    r = np.rint(x / spacing) * spacing          # np.rint rounds half to even
    big = np.abs(r) > 3.3895313892515355e38     # largest finite bf16 (0x7F7F)
    r = np.where(big, np.copysign(np.inf, x), r)
    return np.where(np.isfinite(x), r, x)


def _rounder(dtype):
    return round_bf16 if dtype == BF16 else (lambda a: a)


# ----------------------------------------------------------------------------- elementwise

def silu(z):
    """SiLU(z) = z * sigmoid(z)."""
    return z / (1.0 + np.exp(-z))


def gelu_tanh(z):
    """tanh approximation of GELU: z/2 * (1 + tanh(sqrt(2/pi) (z + 0.044715 z^3)))."""
    return 0.5 * z * (1.0 + np.tanh(math.sqrt(2.0 / math.pi) * (z + 0.044715 * z ** 3)))


def layer_norm(x, eps):
    """LayerNorm over the last axis, no affine, biased variance."""
    mu = x.mean(axis=-1, keepdims=True)
    var = ((x - mu) ** 2).mean(axis=-1, keepdims=True)
    return (x - mu) / np.sqrt(var + eps)


def rms_norm(x, g, eps):
    """x * g / sqrt(mean(x^2) + eps) over the last axis."""
    return x * g / np.sqrt((x ** 2).mean(axis=-1, keepdims=True) + eps)


def softmax(s):
    """Softmax over the last axis (shifted by the row maximum, which leaves it unchanged)."""
    e = np.exp(s - s.max(axis=-1, keepdims=True))
    return e / e.sum(axis=-1, keepdims=True)


def attention(q, k, v):
    """softmax(q k^T / sqrt(d)) v for each (batch, head); q [B,H,Nq,d], k,v [B,H,N,d].
    Computed one (batch, head) pair at a time to bound memory."""
    B, H, Nq, d = q.shape
    out = np.empty((B, H, Nq, v.shape[-1]), dtype=np.float64)
    for b in range(B):
        for h in range(H):
            s = q[b, h] @ k[b, h].T / math.sqrt(d)
            out[b, h] = softmax(s) @ v[b, h]
    return out


# ----------------------------------------------------------------------------- conditioning

def timestep_embedding(s, dim=TEMB_DIM):
    """Sinusoidal embedding [cos(s f_k)]_{k<dim/2} ++ [sin(s f_k)]_{k<dim/2},
    f_k = exp(-ln(10^4) k / (dim/2))  (the DiT time embedder)."""
    half = dim // 2
    f = np.exp(-math.log(10000.0) * np.arange(half, dtype=np.float64) / half)
    return np.concatenate([np.cos(s * f), np.sin(s * f)])


def conditioning(c, t, G):
    """c_t = c + W_t2 SiLU(W_t1 phi(1000 t) + b_t1) + b_t2; c [B,C] -> [B,C]."""
    phi = timestep_embedding(1000.0 * t)
    h1 = silu(_f64(G["t1_w"]) @ phi + _f64(G["t1_b"]))
    temb = _f64(G["t2_w"]) @ h1 + _f64(G["t2_b"])
    return _f64(c) + temb[None, :]


def _f64(a):
    return np.asarray(a, dtype=np.float64)


# ----------------------------------------------------------------------------- (un)patchify

def patchify(x, patch):
    """x [B, C_lat, F, H, W] -> [B, N_img, pt*ph*pw*C_lat].  Tokens in (f, y, x) row-major
    order; features in (channel, dt, dy, dx) order (a strided-convolution patch embed)."""
    B, C, F, H, W = x.shape
    pt, ph, pw = patch
    y = x.reshape(B, C, F // pt, pt, H // ph, ph, W // pw, pw)
    y = y.transpose(0, 2, 4, 6, 1, 3, 5, 7)
    return y.reshape(B, (F // pt) * (H // ph) * (W // pw), C * pt * ph * pw)


def unpatchify(y, patch, lat):
    """Inverse token layout for the model output: y [B, N_img, pt*ph*pw*C_lat] with
    features in (dt, dy, dx, channel) order -> [B, C_lat, F, H, W]."""
    C, F, H, W = lat
    pt, ph, pw = patch
    B = y.shape[0]
    z = y.reshape(B, F // pt, H // ph, W // pw, pt, ph, pw, C)
    z = z.transpose(0, 7, 1, 4, 2, 5, 3, 6)
    return z.reshape(B, C, F, H, W)


# ----------------------------------------------------------------------------- blocks (Eq. 1)

def _heads(x, H):
    """[B, N, H*d] -> [B, H, N, d]; column h*d + e is head h, element e."""
    B, N, C = x.shape
    return x.reshape(B, N, H, C // H).transpose(0, 2, 1, 3)


def _merge(x):
    """[B, H, N, d] -> [B, N, H*d]."""
    B, H, N, d = x.shape
    return x.transpose(0, 2, 1, 3).reshape(B, N, H * d)


def _linear(a, w, b):
    """a W^T + b with W stored [out, in]."""
    return a @ _f64(w).T + _f64(b)


def _rows(rows, n):
    return np.arange(n) if rows is None else np.asarray(rows)


def dit_block(u, cs, W, cfg, rows=None):
    """DiT block with adaLN-Zero style modulation (Peebles & Xie):
      [a1,b1,g1,a2,b2,g2] = SiLU(c_t) W_mod^T + b_mod
      x1 = u + g1 * (Attn(LN(u)(1+b1)+a1) W_o^T + b_o)
      h  = x1 + g2 * (GELU_tanh((LN(x1)(1+b2)+a2) W_1^T + b_1) W_2^T + b_2)
    u [B,N,C] fp64; cs = SiLU(c_t) [B,C].  Returns h for token rows `rows` (all if None):
    attention for a query row needs every key/value row but nothing else of other rows."""
    C, H, eps = cfg["C"], cfg["H"], cfg["ln_eps"]
    r = _rows(rows, u.shape[1])
    mod = _linear(cs, W["mod_w"], W["mod_b"])
    a1, b1, g1, a2, b2, g2 = [m[:, None, :] for m in np.split(mod, 6, axis=-1)]
    a = layer_norm(u, eps) * (1.0 + b1) + a1
    qkv = _linear(a, W["qkv_w"], W["qkv_b"])
    q, k, v = qkv[..., :C], qkv[..., C:2 * C], qkv[..., 2 * C:]
    att = _merge(attention(_heads(q[:, r], H), _heads(k, H), _heads(v, H)))
    x1 = u[:, r] + g1 * _linear(att, W["o_w"], W["o_b"])
    m = layer_norm(x1, eps) * (1.0 + b2) + a2
    return x1 + g2 * _linear(gelu_tanh(_linear(m, W["fc1_w"], W["fc1_b"])), W["fc2_w"], W["fc2_b"])


def rope_positions(cfg):
    """Position ids [N, 3] of a sample's rows for rotary embedding (FLUX-style 3-axis ids;
    reading where the configs are silent): (0, 0, 0) for text rows, (frame, row, column)
    of the image row's patch in the (F/pt, H/ph, W/pw) grid."""
    _, F, Hh, Wd = cfg["lat"]
    pt, ph, pw = cfg["patch"]
    Fp, Hp, Wp = F // pt, Hh // ph, Wd // pw
    nt = cfg["n_txt"]
    pos = np.zeros((nt + Fp * Hp * Wp, 3))
    t = np.arange(Fp * Hp * Wp)
    pos[nt:, 0] = t // (Hp * Wp)
    pos[nt:, 1] = (t // Wp) % Hp
    pos[nt:, 2] = t % Wp
    return pos


def rope(x, pos, axes, theta):
    """Rotary position embedding of per-head vectors x [B, H, N, d]: the d dims are split
    into consecutive chunks of axes[0], axes[1], axes[2] dims; in chunk a the pair
    (2i, 2i+1) is turned by the angle pos[n, a] * theta^(-2i / axes[a])."""
    out = np.array(x, dtype=np.float64, copy=True)
    start = 0
    for a, da in enumerate(axes):
        if da == 0:
            continue
        i = np.arange(da // 2)
        ang = pos[:, a][:, None] * (float(theta) ** (-2.0 * i / da))[None, :]   # [N, da/2]
        c, sn = np.cos(ang), np.sin(ang)
        x0, x1 = x[..., start + 2 * i], x[..., start + 2 * i + 1]
        out[..., start + 2 * i] = x0 * c - x1 * sn
        out[..., start + 2 * i + 1] = x0 * sn + x1 * c
        start += da
    return out


def _qk_rope(q, k, cfg):
    """q, k after their RMS norms, rotated when the model has rotary axes (rope_axes)."""
    axes = cfg.get("rope_axes", (0, 0, 0))
    if not sum(axes):
        return q, k
    pos = rope_positions(cfg)
    th = cfg.get("rope_theta", 10000.0)
    return rope(q, pos, axes, th), rope(k, pos, axes, th)


def double_block(u, cs, W, cfg, rows=None):
    """MMDiT double-stream block (SD3 / FLUX style): text rows [0, n_txt) and image rows
    [n_txt, N) of each sample carry their own DiT weight sets; q and k are RMS-normalised
    per head with learned gains; attention is joint over all N rows; each stream then
    applies its own output projection, gated residual and MLP exactly as in dit_block."""
    C, H, d, eps = cfg["C"], cfg["H"], cfg["d"], cfg["ln_eps"]
    nt = cfg["n_txt"]
    N = u.shape[1]
    r = _rows(rows, N)
    seg = {"txt": slice(0, nt), "img": slice(nt, N)}
    mods, qs, ks, vs = {}, [], [], []
    for s in ("txt", "img"):
        Ws = W[s]
        mod = _linear(cs, Ws["mod_w"], Ws["mod_b"])
        mods[s] = [m[:, None, :] for m in np.split(mod, 6, axis=-1)]
        a1, b1 = mods[s][0], mods[s][1]
        a = layer_norm(u[:, seg[s]], eps) * (1.0 + b1) + a1
        qkv = _linear(a, Ws["qkv_w"], Ws["qkv_b"])
        qs.append(rms_norm(_heads(qkv[..., :C], H), _f64(Ws["q_g"]), eps))
        ks.append(rms_norm(_heads(qkv[..., C:2 * C], H), _f64(Ws["k_g"]), eps))
        vs.append(_heads(qkv[..., 2 * C:], H))
    q, k = _qk_rope(np.concatenate(qs, axis=2), np.concatenate(ks, axis=2), cfg)
    v = np.concatenate(vs, axis=2)
    att = _merge(attention(q[:, :, r], k, v))          # [B, len(r), C]
    out = np.empty((u.shape[0], len(r), C), dtype=np.float64)
    for s in ("txt", "img"):
        sel = (r < nt) if s == "txt" else (r >= nt)
        if not sel.any():
            continue
        Ws = W[s]
        _, _, g1, a2, b2, g2 = mods[s]
        x1 = u[:, r[sel]] + g1 * _linear(att[:, sel], Ws["o_w"], Ws["o_b"])
        m = layer_norm(x1, eps) * (1.0 + b2) + a2
        out[:, sel] = x1 + g2 * _linear(gelu_tanh(_linear(m, Ws["fc1_w"], Ws["fc1_b"])),
                                        Ws["fc2_w"], Ws["fc2_b"])
    return out


def single_block(u, cs, W, cfg, rows=None):
    """MMDiT single-stream block (FLUX style), one weight set over all N rows:
      [a, b, g] = SiLU(c_t) W_mod^T + b_mod
      [q|k|v|z] = (LN(u)(1+b)+a) W_1^T + b_1          (C -> 3C + mlp)
      h = u + g * ([Attn(rms(q), rms(k), v) | GELU_tanh(z)] W_2^T + b_2)   (C + mlp -> C)"""
    C, H, eps = cfg["C"], cfg["H"], cfg["ln_eps"]
    r = _rows(rows, u.shape[1])
    mod = _linear(cs, W["mod_w"], W["mod_b"])
    a_, b_, g_ = [m[:, None, :] for m in np.split(mod, 3, axis=-1)]
    a = layer_norm(u, eps) * (1.0 + b_) + a_
    y = _linear(a, W["lin1_w"], W["lin1_b"])
    q, k = _qk_rope(rms_norm(_heads(y[..., :C], H), _f64(W["q_g"]), eps),
                    rms_norm(_heads(y[..., C:2 * C], H), _f64(W["k_g"]), eps), cfg)
    v = _heads(y[..., 2 * C:3 * C], H)
    att = _merge(attention(q[:, :, r], k, v))
    z = gelu_tanh(y[:, r, 3 * C:])
    return u[:, r] + g_ * _linear(np.concatenate([att, z], axis=-1), W["lin2_w"], W["lin2_b"])


def block(kind, u, cs, W, cfg, rows=None):
    """Exact block output h_f = B_l(u; t, c) (Eq. 1) for the block kind."""
    if kind == DIT:
        return dit_block(u, cs, W, cfg, rows)
    if kind == MMDIT_DOUBLE:
        return double_block(u, cs, W, cfg, rows)
    return single_block(u, cs, W, cfg, rows)


def final_layer(x_img, cs, G, cfg):
    """Final adaLN + linear: [a_f|b_f] = SiLU(c_t) W_fmod^T + b; y = (LN(x)(1+b_f)+a_f) W_f^T + b_f."""
    mod = _linear(cs, G["fmod_w"], G["fmod_b"])
    a_f, b_f = [m[:, None, :] for m in np.split(mod, 2, axis=-1)]
    return _linear(layer_norm(x_img, cfg["ln_eps"]) * (1.0 + b_f) + a_f, G["f_w"], G["f_b"])


# ----------------------------------------------------------------------------- schedule

def make_plan(T, L, R, K, S, mask, mode):
    """Fixed schedule (Sec. 3.3: sites frozen before evaluation; Eq. 2: finite differences
    estimated at exact refreshes).  Readings: refresh at steps i with i mod R == 0 (every
    step in Vanilla); j(i) = number of refreshes up to i minus one; forecast order
    k_eff = min(K, j); the Delta of refresh j lives in ring slot j mod S; at a cached step
    the forecast reads slots (j - m) mod S, m = 0..k_eff.  Site bits on refresh steps are
    ignored.  Verify, FeatFix, Exact-only and the partial arms share one plan; Draft has no
    sites.  The whole-timestep recompute arm (Sec. 3.3: recomputation repeats the
    remaining transformer stack) pays the first site of a cached step and recomputes every
    later layer of that step exactly (RECOMPUTE_ACT, no history refresh)."""
    mask = np.asarray(mask, dtype=np.uint8).reshape(T, L)
    refresh = np.array([mode == VANILLA or i % R == 0 for i in range(T)])
    j = np.cumsum(refresh) - 1
    k_eff = np.minimum(K, j)
    step_kind = np.where(refresh, REFRESH_STEP, CACHED_STEP).astype(np.int32)
    write_slot = np.full(T, -1, np.int32)
    read_slots = np.full((T, K + 1), -1, np.int32)
    action = np.zeros((T, L), np.int32)
    for i in range(T):
        if refresh[i]:
            action[i, :] = EXACT
            if mode != VANILLA:
                write_slot[i] = j[i] % S
        else:
            for m in range(k_eff[i] + 1):
                read_slots[i, m] = (j[i] - m) % S
            paid_seen = False
            for l in range(L):
                if mode == RECOMPUTE and paid_seen:
                    action[i, l] = RECOMPUTE_ACT
                    continue
                paid = mask[i, l] and mode in PAID_MODES
                action[i, l] = SITE if paid else DRAFT_ACT
                paid_seen = paid_seen or paid
    n_site = int((action == SITE).sum())
    counts = {"n_full_refresh": int(refresh.sum()), "n_paid_checks": n_site,
              "n_forwarded": n_site if mode in FORWARDING_MODES else 0,
              "n_recomputed": int((action == RECOMPUTE_ACT).sum())}
    return {"step_kind": step_kind, "refresh_ord": j.astype(np.int32),
            "k_eff": k_eff.astype(np.int32), "read_slots": read_slots,
            "write_slot": write_slot, "action": action, "counts": counts}


def forward_partial(hd, hf, mode, stride):
    """The partial arms (Sec. 3.3, token- and channel-level replacement): the exact output
    at every stride-th token (row of the block, text rows included) or channel, counted
    from 0 within each sample; the draft elsewhere."""
    out = hd.copy()
    if mode == TOKENS_PARTIAL:
        out[:, ::stride, :] = hf[:, ::stride, :]
    else:
        out[:, :, ::stride] = hf[:, :, ::stride]
    return out


class TaylorCache:
    """Per-layer finite-difference history (Eq. 2, TaylorSeer-style estimator).

    At refresh j (step tau_j) with new feature Delta:
        D^0 <- Delta,  D^{k+1} <- (D^k_new - D^k_old) / (tau_j - tau_{j-1}),  k < min(K, j).
    Forecast at step i:  F(i) = sum_{k=0..min(K,j)} (i - tau_j)^k / k! * D^k.
    K = 0 is plain reuse of the last refreshed feature."""

    def __init__(self, K):
        self.K = K
        self.D = []
        self.tau = None
        self.j = -1

    def refresh(self, delta, tau):
        j = self.j + 1
        new = [delta]
        for k in range(min(self.K, j)):
            new.append((new[k] - self.D[k]) / (tau - self.tau))
        self.D, self.tau, self.j = new, tau, j

    def forecast(self, i):
        if self.j < 0:
            raise RuntimeError("forecast before the first refresh")
        m = i - self.tau
        k_eff = min(self.K, self.j)
        out = 0.0
        for k in range(k_eff + 1):
            out = out + (m ** k / math.factorial(k)) * self.D[k]
        return out


def rel_l1(hd, hf, eps):
    """Eq. 4 per sample b: sum|hd - hf| / (sum|hf| + eps) over that sample's N*C elements."""
    B = hf.shape[0]
    num = np.abs(hd - hf).reshape(B, -1).sum(axis=1)
    den = np.abs(hf).reshape(B, -1).sum(axis=1)
    return num / (den + eps)


# ----------------------------------------------------------------------------- the loop

def run(cfg, mode, inputs, weights, mask, feature_mode=RESIDUAL, trace=None, tau=0.0, stride=2):
    """Whole cached denoising loop (Sec. 3.3 framework, Eq. 1-5).

    Sampler reading: rectified-flow Euler on t_i = 1 - i/T, x_{i+1} = x_i + (t_{i+1}-t_i) v.
    Precision reading: fp64 throughout; in bf16 workloads values are rounded to bf16 where
    the GPU stores them between layers: the stream after each layer (and after the patch
    embedding), and each cached Delta.

    tau > 0 (Verify and FeatFix) replaces the fixed refresh rule by an adaptive base
    policy (Sec. 3.1: the base policy decides when to refresh; Sec. 4: the FLUX policy
    has a threshold).  Reading: step 0 refreshes; step i refreshes when R steps have
    passed since the last refresh, or when step i-1 was a cached step with paid sites
    whose largest discrepancy over those sites and the samples (Eq. 4) is not <= tau
    (NaN counts as above).  Sites keep the mask; the finite differences use the actual
    refresh steps (Eq. 2).

    Classifier-free guidance (cfg["cfg_pairs"] = 1; reading of the usual batch doubling):
    the B model rows are B/2 conditional samples and their B/2 unconditional twins (rows
    b and B/2 + b, conditioned by inputs["c"] / inputs["txt"] rows); both read latent b of
    x ([B/2, ...]), and the Euler step uses v = v_u + s (v_c - v_u), s = cfg["cfg_scale"].

    The matched-compute arms (Sec. 3.3) differ from FeatFix only at paid sites: the token
    and channel arms forward the exact output on every `stride`-th token or channel
    (forward_partial); the recompute arm forwards it and runs the rest of the step exact.

    Returns dict(x=x_T [fp64], audit={(i, l): d[B]}, counts, plan, step_kind=[T]).  If
    `trace` is a list, the stream after every (step, layer) is appended to it."""
    T, R, K, S = cfg["T"], cfg["R"], cfg["K"], cfg["S"]
    kinds = cfg["kinds"]
    L = len(kinds)
    rnd = _rounder(cfg["dtype"])
    layer_w, G = weights
    plan = make_plan(T, L, R, K, S, mask, mode)
    if tau > 0 and mode not in (VERIFY, FEATFIX):
        raise ValueError("tau > 0 needs the discrepancy of Verify or FeatFix")
    site_mask = np.asarray(mask, dtype=np.uint8).reshape(T, L)
    x = _f64(inputs["x"]).copy()
    txt = _f64(inputs["txt"])
    n_txt = cfg["n_txt"]
    caches = [TaylorCache(K) for _ in range(L)]
    audit = {}
    step_kind = []
    counts = {"n_full_refresh": 0, "n_paid_checks": 0, "n_forwarded": 0, "n_recomputed": 0}
    last, prev_d = -1, None   # last refresh step; largest site discrepancy of the previous step
    for i in range(T):
        if tau > 0:
            refresh = i == 0 or i - last >= R or (prev_d is not None and not prev_d <= tau)
            actions = [EXACT] * L if refresh else [SITE if site_mask[i, l] else DRAFT_ACT for l in range(L)]
        else:
            refresh = plan["step_kind"][i] == REFRESH_STEP
            actions = plan["action"][i]
        if refresh:
            last = i
            counts["n_full_refresh"] += 1
        step_kind.append(REFRESH_STEP if refresh else CACHED_STEP)
        step_d = []
        t_i, t_n = 1.0 - i / T, 1.0 - (i + 1) / T
        cs = silu(conditioning(inputs["c"], t_i, G))
        pt = patchify(x, cfg["patch"])
        if cfg.get("cfg_pairs"):
            pt = np.concatenate([pt, pt], axis=0)      # rows b and B/2 + b read latent b
        X = rnd(_linear(pt, G["pe_w"], G["pe_b"]))
        if n_txt:
            X = np.concatenate([txt, X], axis=1)
        for l in range(L):
            act = actions[l]
            u = X
            if act == EXACT:
                h = rnd(block(kinds[l], u, cs, layer_w[l], cfg))
                if mode != VANILLA:
                    caches[l].refresh(rnd(h - u) if feature_mode == RESIDUAL else h, i)
                X = h
            elif act == RECOMPUTE_ACT:
                counts["n_recomputed"] += 1
                X = rnd(block(kinds[l], u, cs, layer_w[l], cfg))
            else:
                F = caches[l].forecast(i)
                hd = rnd(u + F) if feature_mode == RESIDUAL else rnd(F)
                if act == DRAFT_ACT:
                    X = hd
                else:
                    counts["n_paid_checks"] += 1
                    hf = rnd(block(kinds[l], u, cs, layer_w[l], cfg))
                    if mode != EXACT_ONLY:
                        audit[(i, l)] = rel_l1(hd, hf, cfg["rel_eps"])
                        step_d.append(audit[(i, l)])
                    if mode in FORWARDING_MODES:
                        counts["n_forwarded"] += 1
                    if mode in (TOKENS_PARTIAL, CHANNELS_PARTIAL):
                        X = forward_partial(hd, hf, mode, stride)
                    else:
                        X = hf if mode in (FEATFIX, EXACT_ONLY, RECOMPUTE) else hd
            if trace is not None:
                trace.append(X.copy())
        prev_d = float(np.max(np.concatenate(step_d))) if step_d else None
        y = final_layer(X[:, n_txt:], cs, G, cfg)
        v = unpatchify(y, cfg["patch"], cfg["lat"])
        if cfg.get("cfg_pairs"):
            half = v.shape[0] // 2
            v = v[half:] + cfg["cfg_scale"] * (v[:half] - v[half:])
        x = x + (t_n - t_i) * v
    return {"x": x, "audit": audit, "counts": counts, "plan": plan, "step_kind": step_kind}


def max_rel_err(a, b):
    """Normwise max relative error max|a - b| / max|b| (b is the reference)."""
    a = np.asarray(a, dtype=np.float64)
    b = np.asarray(b, dtype=np.float64)
    return float(np.abs(a - b).max() / np.abs(b).max())


def block_flops(cfg, kind):
    """Algorithmic FLOPs of one exact block (GEMMs 2*M*N*K each, attention 4*B*N^2*C)."""
    B, C, M = cfg["B"], cfg["C"], cfg["mlp"]
    N = cfg["n_img"] + cfg["n_txt"]
    rows = B * N
    if kind == MMDIT_SINGLE:
        lin = 2 * rows * C * (3 * C + M) + 2 * rows * (C + M) * C
    else:
        lin = 2 * rows * C * (3 * C + C + M + M)
    return lin + 4 * B * N * N * C
