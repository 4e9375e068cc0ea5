"""Seeded synthetic inputs for the segmented gated linear recurrence and the
short convolution.

This module only draws random numbers in the shapes and distributions of the
workloads; it holds none of the recurrence's arithmetic, so both the HIP path
and the CPU oracle may take their inputs from it.

Recipe (every workload):
  * draw order q, k, v, x_g, S_in, dO, dS_out from one torch.Generator seeded
    with `seed`, all in float32;
  * q, v, dO ~ N(0, 1); k ~ N(0, 1) then L2-normalised over its channel dim;
  * g = log(sigmoid(x_g)) with x_g ~ N(g_mu, 1) (natural-log decay, float32),
    one value per (token, head) for the scalar gate, one per key channel for the
    vector gate;
  * S_in ~ s_in_std * N(0, 1) (zero when s_in_std == 0); dS_out likewise;
  * q, k, v, dO are then rounded (round-to-nearest-even) to the I/O dtype.
"""
import torch

# Workload shapes of the paper's evaluation (Sec. 4.1: a 15B-class GDN layer has
# hidden 5120 = 40 heads x 128; the 256K context is the longest the paper runs).
WORKLOADS = {
    # tiny fp32 parity case: one 1024-token segment, d = 64
    "tiny_fp32": dict(B=1, H=2, D=64, seg_lens=[1024], io="f32", gate="scalar",
                      g_mu=3.0, s_in_std=0.0),
    # mid layer: 32K tokens in 8 uniform segments, bf16 I/O, nonzero initial state
    "mid_bf16": dict(B=1, H=16, D=128, seg_lens=[4096] * 8, io="bf16", gate="scalar",
                     g_mu=3.0, s_in_std=0.1),
    # 256K-context shard, 40 heads of 128, 8 nonuniform segments
    "ctx256k_h40": dict(B=1, H=40, D=128,
                        seg_lens=[65536, 40960, 32768, 28672, 26624, 24576, 22528, 20480],
                        io="bf16", gate="scalar", g_mu=3.0, s_in_std=0.0),
    # GLA-style per-key-channel gate
    "vector_gate": dict(B=2, H=16, D=128, seg_lens=[4096] * 16, io="bf16", gate="vector",
                        g_mu=3.0, s_in_std=0.0),
    # many short segments with stronger decay: exposes the state transitions
    "scan_stress": dict(B=4, H=32, D=128, seg_lens=[512] * 32, io="bf16", gate="scalar",
                        g_mu=1.0, s_in_std=0.0),
}

_IO = {"f32": torch.float32, "bf16": torch.bfloat16}


def workload(name, **override):
    w = dict(WORKLOADS[name])
    w.update(override)
    w["name"] = name
    return w


def make_inputs(w, device="cpu", seed=1000, dS_out_std=0.0, L=None):
    """Draw one set of inputs for workload dict `w` on `device`.

    L (optional) truncates the sequence to its first L tokens (the draws are
    made at the truncated size, so a truncated set is not a prefix of the full
    one).  Returns a dict with q, k, v, dO (I/O dtype, [B, L, H, D]), g
    (float32, [B, L, H] or [B, L, H, D]), S_in and dS_out (float32
    [B, H, D, D] or None) and seg_lens.
    """
    B, H, D = w["B"], w["H"], w["D"]
    seg_lens = list(w["seg_lens"])
    if L is None:
        L = sum(seg_lens)
    else:
        seg_lens = [L]
    io = _IO[w["io"]]
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    f32 = dict(dtype=torch.float32, device=device, generator=gen)

    def randn(*shape):
        return torch.randn(*shape, **f32)

    q = randn(B, L, H, D)
    k = randn(B, L, H, D)
    k = k / k.norm(dim=-1, keepdim=True)
    v = randn(B, L, H, D)
    gshape = (B, L, H, D) if w["gate"] == "vector" else (B, L, H)
    xg = randn(*gshape) + float(w["g_mu"])
    g = torch.nn.functional.logsigmoid(xg)
    del xg
    S_in = randn(B, H, D, D) * float(w["s_in_std"]) if w["s_in_std"] > 0 else None
    dO = randn(B, L, H, D)
    dS_out = randn(B, H, D, D) * float(dS_out_std) if dS_out_std > 0 else None
    out = dict(q=q.to(io), k=k.to(io), v=v.to(io), g=g.contiguous(), S_in=S_in,
               dO=dO.to(io), dS_out=dS_out, seg_lens=seg_lens)
    return out


# Short convolution in front of the recurrence (GDN-style: 4 taps, SiLU) over the
# q, k and v projections of the 256K-context layer: 3 x 40 x 128 channels, the
# same 8 segments, tails carried from segment to segment.
CONV_WORKLOADS = {
    "conv_ctx256k": dict(B=1, C=3 * 40 * 128, W=4, seg_lens=WORKLOADS["ctx256k_h40"]["seg_lens"], io="bf16",
                         act="silu"),
}


def conv_workload(name, **override):
    w = dict(CONV_WORKLOADS[name])
    w.update(override)
    w["name"] = name
    return w


def make_conv_inputs(B, L, C, W, io="bf16", device="cpu", seed=2000, tails=True):
    """Draws, in this order, from one torch.Generator seeded with `seed`:
    x ~ N(0, 1) [B, L, C]; w ~ N(0, 1/W) [C, W]; tail_in ~ N(0, 1) [B, W-1, C];
    dy ~ N(0, 1) [B, L, C]; dtail_out ~ N(0, 1) [B, W-1, C].  x, dy and the
    tail (which holds earlier inputs) are rounded to the I/O dtype; w and the
    tails are float32.  tails=False gives tail_in = dtail_out = None."""
    io_t = _IO[io]
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    f32 = dict(dtype=torch.float32, device=device, generator=gen)
    x = torch.randn(B, L, C, **f32).to(io_t)
    w = (torch.randn(C, W, **f32) / float(W) ** 0.5).contiguous()
    tail_in = torch.randn(B, W - 1, C, **f32).to(io_t).float() if W > 1 else None
    dy = torch.randn(B, L, C, **f32).to(io_t)
    dtail_out = torch.randn(B, W - 1, C, **f32) if W > 1 else None
    if not tails:
        tail_in = dtail_out = None
    return dict(x=x, w=w, tail_in=tail_in, dy=dy, dtail_out=dtail_out)


def make_gdn_inputs(B, L, H, D, device="cpu", seed=4000, s_in_std=0.1, g_mu=3.0, key_spread=None, beta_min=0.0):
    """Gated-delta-rule inputs, drawn in this order from one generator seeded
    with `seed`: q, k, v ~ N(0, 1) [B, L, H, D] (k then L2-normalised per
    token, as the delta rule assumes); x_g ~ N(g_mu, 1) and g = log(sigmoid(x_g));
    x_b ~ N(0, 1) and beta = sigmoid(x_b) [B, L, H]; S_in ~ s_in_std * N(0, 1)
    [B, H, D, D] (None when s_in_std == 0).  q, k, v are rounded to bf16; g,
    beta and S_in are float32.

    Nearly parallel keys (key_spread set): then one more draw, a direction
    u ~ N(0, 1) [B, 1, H, D] per head, and k = normalise(u / |u| + key_spread *
    k) with k the normalised draw above.  beta_min > 0 maps beta into
    [beta_min, 1) (beta_min + (1 - beta_min) beta).  Neither changes the draws
    above."""
    gen = torch.Generator(device=device)
    gen.manual_seed(seed)
    f32 = dict(dtype=torch.float32, device=device, generator=gen)
    q = torch.randn(B, L, H, D, **f32)
    k = torch.randn(B, L, H, D, **f32)
    k = k / k.norm(dim=-1, keepdim=True)
    v = torch.randn(B, L, H, D, **f32)
    g = torch.nn.functional.logsigmoid(torch.randn(B, L, H, **f32) + float(g_mu)).contiguous()
    beta = torch.sigmoid(torch.randn(B, L, H, **f32)).contiguous()
    S_in = torch.randn(B, H, D, D, **f32) * float(s_in_std) if s_in_std > 0 else None
    if key_spread is not None:
        u = torch.randn(B, 1, H, D, **f32)
        k = u / u.norm(dim=-1, keepdim=True) + float(key_spread) * k
        k = k / k.norm(dim=-1, keepdim=True)
    if beta_min > 0:
        beta = (float(beta_min) + (1.0 - float(beta_min)) * beta).contiguous()
    return dict(q=q.to(torch.bfloat16), k=k.to(torch.bfloat16), v=v.to(torch.bfloat16), g=g, beta=beta, S_in=S_in)
