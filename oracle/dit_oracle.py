"""Plain CPU oracle for one Diffusion-Transformer denoising step.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: only the tests, the smoke check and the CPU-baseline leg
of the benchmark use it.  It shares no code with the HIP library.

What it computes
----------------
The paper (TetriServe, arXiv 2510.01565) schedules denoising steps of
FLUX.1-dev / SD3 class Diffusion Transformers (Introduction and section 2.1
"DiT Background") but never writes the step's arithmetic down; it only fixes
the number of image tokens per resolution (section 2.2, Table 1; section 6.1
"Workload and Dataset": L = H*W/16^2).  The step below is therefore the plain
definition of an MMDiT denoising step as the models the paper cites define
it: adaLN-modulated LayerNorm, a QKV projection with 2-D rotary position
embedding on image tokens, joint text+image softmax attention, a GELU MLP,
gated residuals, a final adaLN layer that predicts the flow-matching velocity,
and the Euler update x' = x - dt*v.  Every point where the sources leave the
arithmetic open is taken in one documented reading (listed in the design
notes of the repository, items s1..s19):

* LayerNorm: biased variance, eps 1e-6, no affine parameters (s4).
* adaLN: mod(u; shift, scale) = LN(u) * (1 + scale) + shift; modulation
  vector m = W_m SiLU(c) + b_m split in H-wide chunks in the order
  (shift1, scale1, gate1, shift2, scale2, gate2) for double-stream blocks,
  (shift, scale, gate) for single-stream blocks, (shift, scale) for the
  final layer (s3).
* c = W_t2 SiLU(W_t1 e(t) + b_t1) + b_t2 with e(t) the 256-wide sinusoid of
  1000*t, max period 1e4, [cos | sin] order (s5, s6).
* 2-D RoPE: head dims [0, d/2) rotate by the grid row i, [d/2, d) by the grid
  column j; inside an axis slice of width d_a, pair k = (2k, 2k+1) rotates by
  pos * theta^(-2k/d_a), theta = 1e4; text tokens are not rotated (s8).
* Attention: softmax(Q K^T / sqrt(d)) V over the joint sequence [text; image]
  of one request, non-causal (s11).
* GELU: tanh form 0.5 z (1 + tanh(sqrt(2/pi) (z + 0.044715 z^3))) (s10).

Every function works in the precision given by ``dtype`` (float64 unless the
caller asks otherwise); nothing is blocked, fused or reordered beyond the
definitions.  Requests never interact, so a packed batch is the list of its
requests, each stepped on its own.
"""
from __future__ import annotations

from dataclasses import dataclass
from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

F64 = np.float64


# --------------------------------------------------------------------------
# configuration and parameter set
# --------------------------------------------------------------------------
@dataclass(frozen=True)
class OracleConfig:
    """Model shape.  ``tie_streams``: the double-stream blocks use one weight
    set for both streams (a plain joint adaLN DiT block, reading s2)."""
    hidden: int
    heads: int
    head_dim: int
    mlp_ratio: int = 4
    n_double: int = 0
    n_single: int = 0
    in_channels: int = 64
    text_dim: int = 4096
    time_freq_dim: int = 256
    tie_streams: bool = False
    rope_theta: float = 10000.0
    ln_eps: float = 1e-6

    @property
    def mlp_hidden(self) -> int:
        return self.mlp_ratio * self.hidden


def image_tokens(resolution: int, vae_factor: int = 8, patch: int = 2) -> int:
    """Latent image tokens of a square image (section 2.2, Table 1; section 6.1
    gives L_i = H_i * W_i / 16^2, i.e. VAE factor 8 times patch 2)."""
    side = resolution // (vae_factor * patch)
    return side * side


def streams(cfg: OracleConfig) -> Tuple[str, ...]:
    return ("img",) if cfg.tie_streams else ("img", "txt")


def stream_prefix(cfg: OracleConfig, block: int, stream: str) -> str:
    s = "img" if cfg.tie_streams else stream
    return f"double.{block}.{s}."


def modulation_layout(cfg: OracleConfig) -> Dict[str, Tuple[int, int]]:
    """Row offset and chunk count of every adaLN modulation inside the one
    concatenated modulation weight ``mod.w`` [rows, H]: double blocks (img,
    then txt unless tied) with 6 chunks, single blocks with 3, final with 2."""
    H = cfg.hidden
    out: Dict[str, Tuple[int, int]] = {}
    off = 0
    for i in range(cfg.n_double):
        for s in streams(cfg):
            out[f"double.{i}.{s}"] = (off, 6)
            off += 6 * H
    for i in range(cfg.n_single):
        out[f"single.{i}"] = (off, 3)
        off += 3 * H
    out["final"] = (off, 2)
    off += 2 * H
    out["_rows"] = (off, 0)
    return out


def param_shapes(cfg: OracleConfig) -> List[Tuple[str, Tuple[int, ...]]]:
    """Names and shapes of every parameter, Linear weights as [out, in]."""
    H, F, T = cfg.hidden, cfg.mlp_hidden, cfg.time_freq_dim
    mod_rows = modulation_layout(cfg)["_rows"][0]
    p: List[Tuple[str, Tuple[int, ...]]] = [
        ("time_in.w1", (H, T)), ("time_in.b1", (H,)),
        ("time_in.w2", (H, H)), ("time_in.b2", (H,)),
        ("img_in.w", (H, cfg.in_channels)), ("img_in.b", (H,)),
        ("txt_in.w", (H, cfg.text_dim)), ("txt_in.b", (H,)),
        ("mod.w", (mod_rows, H)), ("mod.b", (mod_rows,)),
    ]
    for i in range(cfg.n_double):
        for s in streams(cfg):
            pre = f"double.{i}.{s}."
            p += [(pre + "qkv.w", (3 * H, H)), (pre + "qkv.b", (3 * H,)),
                  (pre + "proj.w", (H, H)), (pre + "proj.b", (H,)),
                  (pre + "mlp1.w", (F, H)), (pre + "mlp1.b", (F,)),
                  (pre + "mlp2.w", (H, F)), (pre + "mlp2.b", (H,))]
    for i in range(cfg.n_single):
        pre = f"single.{i}."
        p += [(pre + "lin1.w", (3 * H + F, H)), (pre + "lin1.b", (3 * H + F,)),
              (pre + "lin2.w", (H, H + F)), (pre + "lin2.b", (H,))]
    p += [("final.w", (cfg.in_channels, H)), ("final.b", (cfg.in_channels,))]
    return p


# --------------------------------------------------------------------------
# elementary functions
# --------------------------------------------------------------------------
def timestep_embedding(t, dim: int = 256, max_period: float = 10000.0,
                       time_scale: float = 1000.0, dtype=F64) -> np.ndarray:
    """Sinusoidal embedding of the scaled timestep (reading s6): frequencies
    f_j = max_period^(-j/(dim/2)), angle a_j = time_scale * t * f_j, output
    [cos a_0 .. cos a_{dim/2-1}, sin a_0 .. sin a_{dim/2-1}]."""
    half = dim // 2
    j = np.arange(half, dtype=F64)
    freqs = np.exp(-np.log(max_period) * j / half)
    a = time_scale * np.asarray(t, dtype=F64)[..., None] * freqs
    return np.concatenate([np.cos(a), np.sin(a)], axis=-1).astype(dtype)


def silu(x: np.ndarray) -> np.ndarray:
    """SiLU(x) = x * sigmoid(x) = x / (1 + exp(-x))."""
    with np.errstate(over="ignore"):
        return x / (1.0 + np.exp(-x))


def gelu_tanh(x: np.ndarray) -> np.ndarray:
    """GELU, tanh approximation (reading s10)."""
    c = np.sqrt(2.0 / np.pi)
    return 0.5 * x * (1.0 + np.tanh(c * (x + 0.044715 * x * x * x)))


def layer_norm(x: np.ndarray, eps: float) -> np.ndarray:
    """Per-row LayerNorm with biased variance and no affine (reading s4)."""
    mu = x.mean(axis=-1, keepdims=True)
    xc = x - mu
    var = (xc * xc).mean(axis=-1, keepdims=True)
    return xc / np.sqrt(var + eps)


def modulate(x: np.ndarray, shift: np.ndarray, scale: np.ndarray, eps: float) -> np.ndarray:
    """adaLN: LN(x) * (1 + scale) + shift (reading s3)."""
    return layer_norm(x, eps) * (1.0 + scale) + shift


def linear(x: np.ndarray, w: np.ndarray, b: Optional[np.ndarray]) -> np.ndarray:
    """y = x W^T + b with W stored [out, in]."""
    y = x @ w.T
    return y if b is None else y + b


def euler_update(x: np.ndarray, v: np.ndarray, dt: float) -> np.ndarray:
    """Flow-matching Euler step: x' = x - dt * v."""
    return x - dt * v


# --------------------------------------------------------------------------
# rotary position embedding (reading s8)
# --------------------------------------------------------------------------
def rope_angles(pos: np.ndarray, axis_dim: int, theta: float) -> np.ndarray:
    """Angles pos * theta^(-2k/axis_dim), k < axis_dim/2, evaluated in fp64.
    Returns [len(pos), axis_dim/2]."""
    k = np.arange(axis_dim // 2, dtype=F64)
    omega = theta ** (-2.0 * k / axis_dim)
    return np.asarray(pos, dtype=F64)[:, None] * omega[None, :]


def rotate_pairs(x: np.ndarray, ang: np.ndarray) -> np.ndarray:
    """Rotate consecutive pairs (2k, 2k+1) of the last axis of x [L, ..., 2P]
    by ang [L, P]: (u, v) -> (u cos - v sin, u sin + v cos)."""
    shape = ang.shape[:1] + (1,) * (x.ndim - 2) + ang.shape[1:]
    c = np.cos(ang).reshape(shape).astype(x.dtype)
    s = np.sin(ang).reshape(shape).astype(x.dtype)
    u, v = x[..., 0::2], x[..., 1::2]
    out = np.empty_like(x)
    out[..., 0::2] = u * c - v * s
    out[..., 1::2] = u * s + v * c
    return out


def rope_2d(x: np.ndarray, grid_h: int, grid_w: int, theta: float) -> np.ndarray:
    """2-D RoPE on image tokens x [h*w, heads, d] in row-major grid order
    (token p sits at row p // w, column p % w)."""
    L, _, d = x.shape
    assert L == grid_h * grid_w and d % 4 == 0
    p = np.arange(L)
    da = d // 2
    out = np.empty_like(x)
    out[..., :da] = rotate_pairs(x[..., :da], rope_angles(p // grid_w, da, theta))
    out[..., da:] = rotate_pairs(x[..., da:], rope_angles(p % grid_w, da, theta))
    return out


# --------------------------------------------------------------------------
# attention (reading s11)
# --------------------------------------------------------------------------
def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray,
              rows: Optional[np.ndarray] = None, q_chunk: int = 2048) -> np.ndarray:
    """O = softmax(Q K^T / sqrt(d)) V per head, exact two-pass softmax
    (row max, exp, divide by the row sum).  q, k, v: [L, heads, d].  ``rows``
    selects query rows (all by default); queries are processed ``q_chunk`` at
    a time only to bound memory, each row's softmax is complete."""
    L, nh, d = k.shape
    qs = q if rows is None else q[rows]
    out = np.empty(qs.shape[:1] + (nh, v.shape[2]), dtype=q.dtype)
    scale = 1.0 / np.sqrt(d)
    for h in range(nh):
        kh, vh = k[:, h, :], v[:, h, :]
        for r0 in range(0, qs.shape[0], q_chunk):
            s = (qs[r0:r0 + q_chunk, h, :] @ kh.T) * scale
            s -= s.max(axis=1, keepdims=True)      # in place: same values, no temporary
            p = np.exp(s)
            p /= p.sum(axis=1, keepdims=True)
            out[r0:r0 + q_chunk, h, :] = p @ vh
    return out


# --------------------------------------------------------------------------
# blocks
# --------------------------------------------------------------------------
def modulation(params: Dict[str, np.ndarray], cfg: OracleConfig, key: str,
               c: np.ndarray, dtype=F64) -> List[np.ndarray]:
    """Chunks of m = W_m SiLU(c) + b_m for modulation ``key`` (reading s3)."""
    off, n = modulation_layout(cfg)[key]
    H = cfg.hidden
    w = params["mod.w"][off:off + n * H].astype(dtype)
    b = params["mod.b"][off:off + n * H].astype(dtype)
    m = linear(silu(np.asarray(c, dtype)), w, b)
    return [m[j * H:(j + 1) * H] for j in range(n)]


def _p(params, name, dtype):
    return params[name].astype(dtype, copy=False)


def double_block(params, cfg: OracleConfig, i: int, x_txt: np.ndarray, x_img: np.ndarray,
                 c: np.ndarray, grid_hw: Tuple[int, int], dtype=F64,
                 rows_txt: Optional[np.ndarray] = None, rows_img: Optional[np.ndarray] = None):
    """Double-stream (MMDiT) block on one request: each stream has its own
    weights and modulation; attention is joint over [text; image].
    ``rows_txt`` / ``rows_img`` select the output rows to compute (all by
    default); keys and values always come from every token."""
    H, nh, d, eps = cfg.hidden, cfg.heads, cfg.head_dim, cfg.ln_eps
    x = {"txt": np.asarray(x_txt, dtype), "img": np.asarray(x_img, dtype)}
    Lt, Li = x["txt"].shape[0], x["img"].shape[0]
    sel = {"txt": np.arange(Lt) if rows_txt is None else np.asarray(rows_txt),
           "img": np.arange(Li) if rows_img is None else np.asarray(rows_img)}
    mkey = {s: f"double.{i}.{'img' if cfg.tie_streams else s}" for s in ("txt", "img")}
    mods = {s: modulation(params, cfg, mkey[s], c, dtype) for s in ("txt", "img")}
    q, k, v = {}, {}, {}
    for s in ("txt", "img"):
        pre = stream_prefix(cfg, i, s)
        sh1, sc1 = mods[s][0], mods[s][1]
        a = modulate(x[s], sh1, sc1, eps)
        y = linear(a, _p(params, pre + "qkv.w", dtype), _p(params, pre + "qkv.b", dtype))
        L = y.shape[0]
        q[s] = y[:, 0:H].reshape(L, nh, d)
        k[s] = y[:, H:2 * H].reshape(L, nh, d)
        v[s] = y[:, 2 * H:3 * H].reshape(L, nh, d)
    gh, gw = grid_hw
    q["img"] = rope_2d(q["img"], gh, gw, cfg.rope_theta)
    k["img"] = rope_2d(k["img"], gh, gw, cfg.rope_theta)
    joint_rows = np.concatenate([sel["txt"], Lt + sel["img"]])
    o = attention(np.concatenate([q["txt"], q["img"]]), np.concatenate([k["txt"], k["img"]]),
                  np.concatenate([v["txt"], v["img"]]), rows=joint_rows)
    o = o.reshape(o.shape[0], H)
    nt = len(sel["txt"])
    o_s = {"txt": o[:nt], "img": o[nt:]}
    out = {}
    for s in ("txt", "img"):
        pre = stream_prefix(cfg, i, s)
        _, _, g1, sh2, sc2, g2 = mods[s]
        xs = x[s][sel[s]]
        xs = xs + g1 * linear(o_s[s], _p(params, pre + "proj.w", dtype), _p(params, pre + "proj.b", dtype))
        hmid = gelu_tanh(linear(modulate(xs, sh2, sc2, eps),
                                _p(params, pre + "mlp1.w", dtype), _p(params, pre + "mlp1.b", dtype)))
        out[s] = xs + g2 * linear(hmid, _p(params, pre + "mlp2.w", dtype), _p(params, pre + "mlp2.b", dtype))
    return out["txt"], out["img"]


def single_block(params, cfg: OracleConfig, i: int, x: np.ndarray, n_txt: int,
                 c: np.ndarray, grid_hw: Tuple[int, int], dtype=F64,
                 rows: Optional[np.ndarray] = None) -> np.ndarray:
    """Single-stream block on one request's joint sequence x = [text; image]:
    one linear produces Q, K, V and the MLP input; attention and GELU(MLP)
    are concatenated and projected by a second linear; one gated residual.
    ``rows`` selects the output rows to compute (all by default)."""
    H, nh, d, eps = cfg.hidden, cfg.heads, cfg.head_dim, cfg.ln_eps
    x = np.asarray(x, dtype)
    L = x.shape[0]
    sel = np.arange(L) if rows is None else np.asarray(rows)
    sh, sc, g = modulation(params, cfg, f"single.{i}", c, dtype)
    pre = f"single.{i}."
    w1, b1 = _p(params, pre + "lin1.w", dtype), _p(params, pre + "lin1.b", dtype)
    a = modulate(x, sh, sc, eps)
    zq = linear(a, w1[:3 * H], b1[:3 * H])          # Q, K, V of every token
    q = zq[:, 0:H].reshape(L, nh, d)
    k = zq[:, H:2 * H].reshape(L, nh, d)
    v = zq[:, 2 * H:3 * H].reshape(L, nh, d)
    gh, gw = grid_hw
    q = np.concatenate([q[:n_txt], rope_2d(q[n_txt:], gh, gw, cfg.rope_theta)])
    k = np.concatenate([k[:n_txt], rope_2d(k[n_txt:], gh, gw, cfg.rope_theta)])
    o = attention(q, k, v, rows=sel).reshape(len(sel), H)
    mlp = gelu_tanh(linear(a[sel], w1[3 * H:], b1[3 * H:]))
    y = linear(np.concatenate([o, mlp], axis=1), _p(params, pre + "lin2.w", dtype), _p(params, pre + "lin2.b", dtype))
    return x[sel] + g * y


def conditioning(params, cfg: OracleConfig, t: float, dtype=F64) -> np.ndarray:
    """c = W_t2 SiLU(W_t1 e(t) + b_t1) + b_t2 (readings s5, s6)."""
    e = timestep_embedding(t, cfg.time_freq_dim, dtype=dtype)
    u = linear(e, _p(params, "time_in.w1", dtype), _p(params, "time_in.b1", dtype))
    return linear(silu(u), _p(params, "time_in.w2", dtype), _p(params, "time_in.b2", dtype))


def final_layer(params, cfg: OracleConfig, x_img: np.ndarray, c: np.ndarray, dtype=F64) -> np.ndarray:
    """Velocity v = mod(x_img; shift_f, scale_f) W_f^T + b_f."""
    sh, sc = modulation(params, cfg, "final", c, dtype)
    return linear(modulate(np.asarray(x_img, dtype), sh, sc, cfg.ln_eps),
                  _p(params, "final.w", dtype), _p(params, "final.b", dtype))


def dit_velocity(params, cfg: OracleConfig, latents: np.ndarray, text: np.ndarray,
                 t: float, grid_hw: Tuple[int, int], dtype=F64, on_block=None) -> np.ndarray:
    """One velocity prediction for one request: latents [h*w, C_in] (patchified,
    row-major grid order), text [L_txt, D_txt] -> v [h*w, C_in].
    ``on_block(depth, x)``, if given, sees the joint hidden state [text; image]
    after every block (depth 0 = after the first block); it only observes."""
    c = conditioning(params, cfg, t, dtype)
    x_img = linear(np.asarray(latents, dtype), _p(params, "img_in.w", dtype), _p(params, "img_in.b", dtype))
    x_txt = linear(np.asarray(text, dtype), _p(params, "txt_in.w", dtype), _p(params, "txt_in.b", dtype))
    for i in range(cfg.n_double):
        x_txt, x_img = double_block(params, cfg, i, x_txt, x_img, c, grid_hw, dtype)
        if on_block is not None:
            on_block(i, np.concatenate([x_txt, x_img]))
    n_txt = x_txt.shape[0]
    x = np.concatenate([x_txt, x_img])
    for i in range(cfg.n_single):
        x = single_block(params, cfg, i, x, n_txt, c, grid_hw, dtype)
        if on_block is not None:
            on_block(cfg.n_double + i, x)
    return final_layer(params, cfg, x[n_txt:], c, dtype)


@dataclass
class OracleRequest:
    """One request of a (possibly packed) batch."""
    grid_h: int
    grid_w: int
    t: float
    latents: np.ndarray   # [grid_h*grid_w, C_in]
    text: np.ndarray      # [L_txt, D_txt]


def dit_step(params, cfg: OracleConfig, requests: Sequence[OracleRequest],
             dt: Sequence[float], dtype=F64) -> Tuple[List[np.ndarray], List[np.ndarray]]:
    """One denoising step of a batch: per request, velocity and Euler-updated
    latents.  Requests do not interact (attention is per request)."""
    vs, xs = [], []
    for r, d_t in zip(requests, dt):
        v = dit_velocity(params, cfg, r.latents, r.text, r.t, (r.grid_h, r.grid_w), dtype)
        vs.append(v)
        xs.append(euler_update(np.asarray(r.latents, dtype), v, d_t))
    return vs, xs

