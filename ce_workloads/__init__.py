"""Seeded synthetic inputs for the CE-Router routed block.

This module only *draws* inputs: hidden states, per-token task flags, sequence
offsets, timesteps, keep ratios and random weights. It holds none of the
routed block's arithmetic (no scoring, no selection, no FFN), so that both the
CPU oracle and the HIP path can be fed from it without sharing any of the
method.

The five named workloads follow the shapes of the paper's two backbones:

* Show-o2-1.5B: hidden size 1536, maximum sequence 1024, a 27x27 = 729 token
  image grid (appendix A.5, Show-o2 architecture table); FFN width 8960.
* BAGEL-7B-MoT: hidden 3584, FFN 18944, two FFN weight sets (understanding /
  generation) in a mixture-of-transformers block (section 4.1).
* M = 4 generation segments (section 4.1, appendix A.2 general table).

Synthetic values stand in for the paper's evaluation suites, which are not
used: hidden ~ N(0, 1), every weight matrix and second-layer vector
~ N(0, 1/d). bf16 workloads round every drawn float32 value to the nearest
bf16 (ties to even), so both sides see the same exactly representable values.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional, Sequence, Tuple

import numpy as np

TOK_GEN = 1   # token belongs to the generation task (core + expansion score)
TOK_KEEP = 2  # token is always retained (text / structure token), never scored

N_SEGMENTS = 4  # M, number of generation expansion scorers


# ----------------------------------------------------------------------------
# bf16 storage helpers (input preparation only)
# ----------------------------------------------------------------------------

def bf16_bits(x: np.ndarray) -> np.ndarray:
    """float32 -> bf16 bit patterns (uint16), round to nearest, ties to even.

    NaN inputs map to a quiet NaN pattern. Used to store drawn inputs. The
    rounding add stays in uint32: it can carry past 2^32 only for NaN bit
    patterns, which are replaced afterwards.
    """
    x = np.ascontiguousarray(x, dtype=np.float32)
    u = x.view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    r = ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)
    nan = np.isnan(x)
    if nan.any():
        r = np.where(nan, ((u >> np.uint32(16)) | np.uint32(0x40)).astype(np.uint16), r)
    return r


def bf16_to_f32(bits: np.ndarray) -> np.ndarray:
    """bf16 bit patterns (uint16) -> float32 values (exact)."""
    b = np.ascontiguousarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return b.view(np.float32)


def bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 values to the nearest bf16 value, returned as float32."""
    return bf16_to_f32(bf16_bits(x))


# ----------------------------------------------------------------------------
# Workload container
# ----------------------------------------------------------------------------

@dataclass
class ScorerWeights:
    """Core scorer (rank r_c) and M expansion scorers (rank r_e each).

    Layouts (row-major):
      w1_core [r_c, d], b1_core [r_c] or None, w2_core [r_c], b2_core float
      w1_exp  [M, r_e, d], b1_exp [M, r_e] or None, w2_exp [M, r_e], b2_exp [M] or None
    Matrices hold dtype-representable float32 values.
    """
    w1_core: np.ndarray
    b1_core: Optional[np.ndarray]
    w2_core: np.ndarray
    b2_core: float
    w1_exp: np.ndarray
    b1_exp: Optional[np.ndarray]
    w2_exp: np.ndarray
    b2_exp: Optional[np.ndarray]

    @property
    def r_core(self) -> int:
        return int(self.w1_core.shape[0])

    @property
    def r_exp(self) -> int:
        return int(self.w1_exp.shape[1])

    @property
    def n_seg(self) -> int:
        return int(self.w1_exp.shape[0])


@dataclass
class FFNWeights:
    """One SwiGLU FFN weight set, nn.Linear layout: gate/up [F, d], down [d, F]."""
    w_gate: np.ndarray
    w_up: np.ndarray
    w_down: np.ndarray


@dataclass
class Workload:
    name: str
    dtype: str                 # "f32" or "bf16"
    seq_offsets: np.ndarray    # int32 [B+1]
    flags: np.ndarray          # uint8 [T]
    t: np.ndarray              # float32 [B]
    keep: np.float32
    hidden: np.ndarray         # float32 [T, d] (bf16-representable when dtype == "bf16")
    scorer: ScorerWeights
    ffn: List[FFNWeights]      # 1 set, or 2 (index = GEN bit) for MoT
    meta: dict = field(default_factory=dict)

    @property
    def B(self) -> int:
        return int(self.seq_offsets.shape[0] - 1)

    @property
    def T(self) -> int:
        return int(self.flags.shape[0])

    @property
    def d(self) -> int:
        return int(self.hidden.shape[1])

    @property
    def d_ff(self) -> int:
        return int(self.ffn[0].w_gate.shape[0])


# ----------------------------------------------------------------------------
# Generators
# ----------------------------------------------------------------------------

def _normal(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    x = rng.standard_normal(size=shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return x


def _cast(x: np.ndarray, dtype: str) -> np.ndarray:
    return bf16_round(x) if dtype == "bf16" else np.ascontiguousarray(x, dtype=np.float32)


def build_layout(segments: Sequence[Sequence[Tuple[int, int]]]) -> Tuple[np.ndarray, np.ndarray]:
    """Per-sequence list of (count, flag) runs -> (seq_offsets int32, flags uint8)."""
    offs = [0]
    flags = []
    for seq in segments:
        n = 0
        for count, flag in seq:
            flags.extend([flag] * int(count))
            n += int(count)
        offs.append(offs[-1] + n)
    return np.asarray(offs, dtype=np.int32), np.asarray(flags, dtype=np.uint8)


def draw_scorer(rng, d, r_c, r_e, dtype, n_seg=N_SEGMENTS, biases=False) -> ScorerWeights:
    std = d ** -0.5
    w1c = _cast(_normal(rng, (r_c, d), std), dtype)
    b1c = _normal(rng, (r_c,), 0.1) if biases else None
    w2c = _normal(rng, (r_c,), std)
    b2c = float(_normal(rng, (1,), 0.1)[0]) if biases else 0.0
    w1e = np.empty((n_seg, r_e, d), dtype=np.float32)
    w2e = np.empty((n_seg, r_e), dtype=np.float32)
    b1e = np.empty((n_seg, r_e), dtype=np.float32) if biases else None
    b2e = np.empty((n_seg,), dtype=np.float32) if biases else None
    for m in range(n_seg):
        w1e[m] = _cast(_normal(rng, (r_e, d), std), dtype)
        if biases:
            b1e[m] = _normal(rng, (r_e,), 0.1)
        w2e[m] = _normal(rng, (r_e,), std)
        if biases:
            b2e[m] = _normal(rng, (1,), 0.1)[0]
    return ScorerWeights(w1c, b1c, w2c, b2c, w1e, b1e, w2e, b2e)


def draw_ffn(rng, d, F, dtype) -> FFNWeights:
    std = d ** -0.5
    wg = _cast(_normal(rng, (F, d), std), dtype)
    wu = _cast(_normal(rng, (F, d), std), dtype)
    wd = _cast(_normal(rng, (d, F), std), dtype)
    return FFNWeights(wg, wu, wd)


def make_workload(name: str, segments, *, d: int, F: int, r_c: int, r_e: int,
                  keep: float, dtype: str, seed, n_sets: int = 1,
                  outlier_frac: float = 0.0, outlier_scale: float = 8.0,
                  t_values: Optional[Sequence[float]] = None,
                  biases: bool = False, n_seg: int = N_SEGMENTS) -> Workload:
    """Generic seeded workload.

    Draw order: hidden, outlier channels, t, scorer (core, then expansions
    m = 0..M-1), FFN weight sets.
    """
    rng = np.random.default_rng(seed)
    seq_offsets, flags = build_layout(segments)
    T = int(flags.shape[0])
    B = int(seq_offsets.shape[0] - 1)
    h = _normal(rng, (T, d), 1.0)
    n_out = int(round(outlier_frac * d))
    out_ch = np.zeros(0, dtype=np.int64)
    if n_out:
        out_ch = np.sort(rng.choice(d, size=n_out, replace=False))
        h[:, out_ch] *= np.float32(outlier_scale)
    hidden = _cast(h, dtype)
    if t_values is None:
        t = rng.random(B, dtype=np.float32)
    else:
        t = np.asarray(t_values, dtype=np.float32).reshape(B)
    scorer = draw_scorer(rng, d, r_c, r_e, dtype, n_seg=n_seg, biases=biases)
    ffn = [draw_ffn(rng, d, F, dtype) for _ in range(n_sets)]
    return Workload(name=name, dtype=dtype, seq_offsets=seq_offsets, flags=flags, t=t,
                    keep=np.float32(keep), hidden=hidden, scorer=scorer, ffn=ffn,
                    meta={"seed": seed, "outlier_channels": out_ch})


# ----------------------------------------------------------------------------
# The five named workloads
# ----------------------------------------------------------------------------

U, G, KEEP = 0, TOK_GEN, TOK_KEEP

CONFIG_NAMES = {
    1: "tiny-understanding-fp32",
    2: "showo2-understanding-bf16",
    3: "showo2-generation-50step-bf16",
    4: "7b-mixed-varlen-bf16",
    5: "bagel-mot-bf16",
}

CONFIG_DESCRIPTIONS = {
    1: "B=1 L=256 (64 text kept + 192 image), d=256, FFN 1024, r_c=64, keep 0.5, fp32",
    2: "B=8 L=1024 (729 image + 295 text kept), d=1536, FFN 8960, r_c=128, keep 0.35, bf16, 2% outlier channels x8",
    3: "B=4 L=4096 latent + 128 text kept, d=1536, FFN 8960, r_c=128 r_e=64, keep 0.5, t = s/49 (50 steps), bf16",
    4: "B=4 varlen (2x[1024 image+256 text], 2x[4096 latent+256 text]), d=3584, FFN 18944, r_c=256 r_e=128, keep 0.4, bf16",
    5: "B=2 L=8192 (4096 und + 4096 gen), MoT 2 FFN sets, d=3584, FFN 18944, r_c=256 r_e=128, keep 0.3, bf16",
}


def config_layout(i: int):
    if i == 1:
        return [[(64, KEEP), (192, U)]]
    if i == 2:
        return [[(729, U), (295, KEEP)]] * 8
    if i == 3:
        return [[(4096, G), (128, KEEP)]] * 4
    if i == 4:
        return [[(1024, U), (256, KEEP)]] * 2 + [[(4096, G), (256, KEEP)]] * 2
    if i == 5:
        return [[(4096, U), (4096, G)]] * 2
    raise ValueError(f"unknown config {i}")


def config_params(i: int) -> dict:
    if i == 1:
        return dict(d=256, F=1024, r_c=64, r_e=32, keep=0.5, dtype="f32")
    if i == 2:
        return dict(d=1536, F=8960, r_c=128, r_e=64, keep=0.35, dtype="bf16",
                    outlier_frac=0.02, outlier_scale=8.0)
    if i == 3:
        return dict(d=1536, F=8960, r_c=128, r_e=64, keep=0.5, dtype="bf16")
    if i == 4:
        return dict(d=3584, F=18944, r_c=256, r_e=128, keep=0.4, dtype="bf16")
    if i == 5:
        return dict(d=3584, F=18944, r_c=256, r_e=128, keep=0.3, dtype="bf16", n_sets=2)
    raise ValueError(f"unknown config {i}")


CONFIG3_STEPS = 50


def config3_t(step: int) -> float:
    """Timestep of denoising step s on config 3's uniform 50-step grid in [0, 1]."""
    return float(np.float32(step) / np.float32(CONFIG3_STEPS - 1))


def make_config(i: int, seed=None, step: Optional[int] = None) -> Workload:
    """Named workload i in 1..5 (seed defaults to i - 1).

    Config 3 is a 50-step generation sweep: `step` picks one step s; the hidden
    states of step s are bf16(h_0 + 0.25 * xi_s), with xi_s drawn from seed
    (2, s), and every sequence uses t = s / 49.
    """
    p = dict(config_params(i))
    if seed is None:
        seed = i - 1
    layout = config_layout(i)
    B = len(layout)
    t_values = None
    if i == 1:
        t_values = [0.0]
    if i == 2:
        t_values = [0.0] * B
    if i == 3:
        s = 0 if step is None else int(step)
        t_values = [config3_t(s)] * B
    w = make_workload(CONFIG_NAMES[i], layout, seed=seed, t_values=t_values, **p)
    if i == 3 and step is not None and step > 0:
        w.hidden = config3_step_hidden(w.hidden, int(step))
        w.meta["step"] = int(step)
    return w


def config3_step_hidden(hidden0: np.ndarray, step: int) -> np.ndarray:
    """Hidden states of config 3's denoising step s from those of step 0:
    bf16(h_0 + 0.25 * xi_s), xi_s standard normal from seed (2, s)."""
    if step == 0:
        return hidden0
    xi = np.random.default_rng([2, int(step)]).standard_normal(size=hidden0.shape, dtype=np.float32)
    return bf16_round(hidden0 + np.float32(0.25) * xi)


def small_workload(kind: str, seed: int = 0, dtype: str = "bf16", **kw) -> Workload:
    """Small shapes spanning several tiles plus ragged tails (for parity tests).

    kinds: "und" (understanding, text kept), "gen" (generation), "mixed"
    (varlen U and G sequences), "mot" (two FFN sets, mixed U/G tokens),
    "interleaved" (U/G/KEEP flags interleaved inside each sequence).
    """
    d = kw.pop("d", 256)
    F = kw.pop("F", 512)
    r_c = kw.pop("r_c", 64)
    r_e = kw.pop("r_e", 32)
    keep = kw.pop("keep", 0.4)
    if kind == "und":
        layout = [[(37, KEEP), (300, U)], [(197, U), (11, KEEP)], [(65, U)]]
        n_sets = 1
    elif kind == "gen":
        layout = [[(400, G), (23, KEEP)], [(129, G), (7, KEEP)], [(1, G)]]
        n_sets = 1
    elif kind == "mixed":
        layout = [[(150, U), (40, KEEP)], [(333, G), (17, KEEP | G)], [(0, U)], [(95, G)],
                  [(3, KEEP)]]
        n_sets = 1
    elif kind == "mot":
        layout = [[(211, U), (190, G)], [(64, G), (77, U), (5, KEEP)]]
        n_sets = 2
    elif kind == "interleaved":
        rng = np.random.default_rng([seed, 77])
        seqs = []
        for L in (257, 130, 64):
            fl = rng.choice([U, G, KEEP, KEEP | G], size=L, p=[0.4, 0.4, 0.1, 0.1])
            seqs.append([(1, int(f)) for f in fl])
        layout = seqs
        n_sets = 2
    else:
        raise ValueError(kind)
    return make_workload(f"small-{kind}", layout, d=d, F=F, r_c=r_c, r_e=r_e, keep=keep,
                         dtype=dtype, seed=seed, n_sets=kw.pop("n_sets", n_sets),
                         biases=kw.pop("biases", True), **kw)


def kept_capacity_upper(flags: np.ndarray, seq_offsets: np.ndarray) -> int:
    """A capacity that always suffices: every token of every sequence."""
    return int(seq_offsets[-1])


def make_drop_pair(segments, keep_t: float, keep_ref: float, noise: float, seed: int):
    """Two timesteps' packed positions over one batch layout, for the drop-set
    stability signals: each routable token draws a random score u; timestep t
    keeps the ceil(keep_t * R) highest u of its sequence, the reference keeps
    the ceil(keep_ref * R) highest of u + noise * v (v another draw), so the two
    drop sets overlap more the smaller the noise. The kept counts are
    round(keep * R) (a generator choice, not the method's rule). Always-kept
    tokens get a position at both timesteps. Returns (seq_offsets, flags, token_pos_t,
    token_pos_ref); positions are plain running counters (only their sign is
    read downstream).
    """
    offs, flags = build_layout(segments)
    rng = np.random.default_rng(seed)
    T = int(offs[-1])
    u = rng.random(T)
    v = rng.random(T)
    tps = []
    for keep, score in ((keep_t, u), (keep_ref, u + noise * v)):
        tp = np.full(T, -1, np.int32)
        pos = 0
        for b in range(len(offs) - 1):
            lo, hi = int(offs[b]), int(offs[b + 1])
            idx = np.arange(lo, hi)
            keep_tok = (flags[lo:hi] & TOK_KEEP) != 0
            routable = idx[~keep_tok]
            n_keep = int(round(keep * len(routable)))  # any count will do for these signals
            chosen = set(routable[np.argsort(-score[routable], kind="stable")[:n_keep]].tolist())
            for i in idx:
                if keep_tok[i - lo] or i in chosen:
                    tp[i] = pos
                    pos += 1
        tps.append(tp)
    return offs, flags, tps[0], tps[1]


def make_attention_inputs(q_lens, kv_lens, n_heads: int, n_kv_heads: int, head_dim: int, seed: int,
                          q_scale: float = 1.0):
    """Packed queries / keys / values for the routed attention: per sequence b,
    q_lens[b] query rows and kv_lens[b] key/value rows, entries N(0,1) (queries
    times q_scale), rounded to bf16. Returns (q [Nq, H, dh], k, v [Nkv, H_kv, dh]
    float32 arrays holding bf16 values, q_offsets, kv_offsets int32)."""
    rng = np.random.default_rng(seed)
    qo = np.concatenate([[0], np.cumsum(q_lens)]).astype(np.int32)
    ko = np.concatenate([[0], np.cumsum(kv_lens)]).astype(np.int32)
    q = bf16_round((rng.standard_normal((int(qo[-1]), n_heads, head_dim)) * q_scale).astype(np.float32))
    k = bf16_round(rng.standard_normal((int(ko[-1]), n_kv_heads, head_dim)).astype(np.float32))
    v = bf16_round(rng.standard_normal((int(ko[-1]), n_kv_heads, head_dim)).astype(np.float32))
    return q, k, v, qo, ko
