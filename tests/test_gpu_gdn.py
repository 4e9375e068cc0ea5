"""GPU parity of the gated-delta-rule forward (sf_gdn_fwd through the C ABI)
against the fp64 oracle (oracle.gdn): o and S_out, bf16 I/O, both head dims,
several chunks with a nonzero initial state, explicit superchunk lengths
(one superchunk, one chunk each, a ragged last superchunk), an empty segment,
no initial state, segments chained through S, and a long segment on sampled
heads."""
import numpy as np
import pytest
import torch

import paper_2608_06838_amd as sf
from oracle import gdn
from paper_2608_06838_amd import synth

from _helpers import assert_close, cores, to64

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def say(msg):
    print(msg, flush=True)


def run(inp, ts=0):
    g = {k: (v.to(DEV) if isinstance(v, torch.Tensor) else v) for k, v in inp.items()}
    o, S = sf.gdn_fwd(g["q"], g["k"], g["v"], g["g"], g["beta"], g["S_in"], ts=ts)
    torch.cuda.synchronize()
    return o, S


def ref(inp, heads=None):
    sel = (lambda x: x) if heads is None else (lambda x: x[:, :, heads])
    S_in = inp["S_in"]
    if S_in is not None and heads is not None:
        S_in = S_in[:, heads]
    return gdn.forward(to64(sel(inp["q"])), to64(sel(inp["k"])), to64(sel(inp["v"])), to64(sel(inp["g"])),
                       to64(sel(inp["beta"])), None if S_in is None else to64(S_in), threads=cores())


@pytest.mark.parametrize("D", [64, 128])
def test_gdn_parity(D):
    """o, S_out and the corrected values V^new."""
    B, L, H = 2, 448, 3
    say(f"[gdn] D={D} B={B} L={L} H={H}")
    inp = synth.make_gdn_inputs(B, L, H, D, seed=4100 + D)
    g = {k: (v.to(DEV) if isinstance(v, torch.Tensor) else v) for k, v in inp.items()}
    o, S, vn = sf.gdn_fwd(g["q"], g["k"], g["v"], g["g"], g["beta"], g["S_in"], with_v_new=True)
    torch.cuda.synchronize()
    o2, S2 = run(inp)
    assert torch.equal(o, o2) and torch.equal(S, S2)
    ro, rS, ru = gdn.forward(*(to64(inp[x]) for x in ("q", "k", "v", "g", "beta", "S_in")), threads=cores(),
                             with_u=True)
    assert_close("o", o, ro, "bf16")
    assert_close("S_out", S, rS, "bf16")
    assert_close("v_new", vn, ru, "bf16")


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("ts", [64, 192, 256, 448])
def test_gdn_superchunks(D, ts):
    """Prep walk ([M | N] per superchunk), fp32 scan over superchunks and the
    output walk from the scanned states, for L = 7 chunks: 448 is one
    superchunk (no prep, no scan), 192 leaves a ragged last superchunk."""
    B, L, H = 1, 448, 3
    say(f"[gdn] superchunks D={D} ts={ts}")
    inp = synth.make_gdn_inputs(B, L, H, D, seed=4500 + D + ts)
    o, S = run(inp, ts)
    ro, rS = ref(inp)
    assert_close("o", o, ro, "bf16")
    assert_close("S_out", S, rS, "bf16")


def test_gdn_no_state_and_empty():
    say("[gdn] no initial state; empty segment")
    inp = synth.make_gdn_inputs(1, 192, 2, 128, seed=4200, s_in_std=0.0)
    o, S = run(inp)
    ro, rS = ref(inp)
    assert_close("o", o, ro, "bf16")
    assert_close("S_out", S, rS, "bf16")
    e = synth.make_gdn_inputs(1, 0, 2, 128, seed=4201)
    _, S0 = run(e)
    assert torch.equal(S0.cpu(), e["S_in"])


def test_gdn_chained_segments():
    """Segments chained through the state equal the oracle over the whole
    sequence."""
    B, H, D = 1, 2, 128
    segs = [256, 64, 320]
    say(f"[gdn] chained {segs}")
    inp = synth.make_gdn_inputs(B, sum(segs), H, D, seed=4300)
    g = {k: (v.to(DEV) if isinstance(v, torch.Tensor) else v) for k, v in inp.items()}
    S, outs, t = g["S_in"], [], 0
    for n in segs:
        o, S = sf.gdn_fwd(g["q"][:, t:t + n], g["k"][:, t:t + n], g["v"][:, t:t + n], g["g"][:, t:t + n],
                          g["beta"][:, t:t + n], S)
        outs.append(o)
        t += n
    torch.cuda.synchronize()
    ro, rS = ref(inp)
    assert_close("o", torch.cat(outs, 1), ro, "bf16")
    assert_close("S_out", S, rS, "bf16")


def test_gdn_long_segment_sampled():
    """16384 tokens (256 chunks) over 8 heads; the oracle runs two of them."""
    B, L, H, D = 1, 16384, 8, 128
    say(f"[gdn] long segment L={L} H={H}")
    inp = synth.make_gdn_inputs(B, L, H, D, seed=4400)
    o, S = run(inp)
    heads = [0, 5]
    ro, rS = ref(inp, heads)
    assert_close("o", o[:, :, heads], ro, "bf16")
    assert_close("S_out", S[:, heads], rS, "bf16")
    assert np.isfinite(to64(o)).all()


# ------------------------------------------------------------------ backward
def run_bwd(inp, dO, dS_out, ts=0):
    g = {k: (v.to(DEV) if isinstance(v, torch.Tensor) else v) for k, v in inp.items()}
    out = sf.gdn_bwd(g["q"], g["k"], g["v"], g["g"], g["beta"], g["S_in"], dO.to(DEV),
                     None if dS_out is None else dS_out.to(DEV), ts=ts)
    torch.cuda.synchronize()
    return out


def ref_bwd(inp, dO, dS_out, heads=None):
    sel = (lambda x: x) if heads is None else (lambda x: x[:, :, heads])
    S_in, dS = inp["S_in"], dS_out
    if heads is not None:
        S_in = None if S_in is None else S_in[:, heads]
        dS = None if dS is None else dS[:, heads]
    return gdn.backward(*(to64(sel(inp[x])) for x in ("q", "k", "v", "g", "beta")),
                        None if S_in is None else to64(S_in), to64(sel(dO)), None if dS is None else to64(dS),
                        threads=cores())


def check_bwd(got, want):
    for name, x, r in zip(("dq", "dk", "dv", "dg", "dbeta", "dS_in"), got, want):
        assert_close(name, x, r, "bf16")


def grads_inputs(inp, seed):
    gen = torch.Generator().manual_seed(seed)
    B, L, H, D = inp["v"].shape
    dO = torch.randn((B, L, H, D), generator=gen).to(torch.bfloat16)
    dS = torch.randn((B, H, D, D), generator=gen) * 0.1
    return dO, dS


@pytest.mark.parametrize("D", [64, 128])
@pytest.mark.parametrize("ts", [0, 192, 448])
def test_gdn_bwd_parity(D, ts):
    """Every gradient against the oracle's hand-written backward; ts = 448 is
    one superchunk, 192 leaves a ragged last one, 0 lets the library choose."""
    B, L, H = 1, 448, 3
    say(f"[gdn bwd] D={D} ts={ts}")
    inp = synth.make_gdn_inputs(B, L, H, D, seed=4600 + D + ts)
    dO, dS = grads_inputs(inp, 4700 + D + ts)
    check_bwd(run_bwd(inp, dO, dS, ts), ref_bwd(inp, dO, dS))


@pytest.mark.parametrize("D", [64, 128])
def test_gdn_nearly_parallel_keys(D):
    """Keys within a few degrees of one direction per head, beta in [0.85, 1),
    decay near 1: (I + A) is far from the identity, and the partial products of
    its inverse grow; forward, V^new and every gradient against the oracle, with
    superchunks (ts = 192)."""
    B, L, H = 1, 448, 2
    say(f"[gdn] nearly parallel keys D={D}")
    inp = synth.make_gdn_inputs(B, L, H, D, seed=5300 + D, g_mu=8.0, key_spread=0.05, beta_min=0.85)
    g = {k: (v.to(DEV) if isinstance(v, torch.Tensor) else v) for k, v in inp.items()}
    o, S, vn = sf.gdn_fwd(g["q"], g["k"], g["v"], g["g"], g["beta"], g["S_in"], ts=192, with_v_new=True)
    torch.cuda.synchronize()
    ro, rS, ru = gdn.forward(*(to64(inp[x]) for x in ("q", "k", "v", "g", "beta", "S_in")), threads=cores(),
                             with_u=True)
    assert_close("o", o, ro, "bf16")
    assert_close("S_out", S, rS, "bf16")
    assert_close("v_new", vn, ru, "bf16")
    dO, dS = grads_inputs(inp, 5400 + D)
    check_bwd(run_bwd(inp, dO, dS, 192), ref_bwd(inp, dO, dS))


def test_gdn_bwd_no_state_and_empty():
    say("[gdn bwd] no S_in, no dS_out; empty segment")
    inp = synth.make_gdn_inputs(2, 192, 2, 128, seed=4800, s_in_std=0.0)
    inp["S_in"] = None
    dO, _ = grads_inputs(inp, 4801)
    check_bwd(run_bwd(inp, dO, None), ref_bwd(inp, dO, None))
    e = synth.make_gdn_inputs(1, 0, 2, 128, seed=4802)
    dO, dS = grads_inputs(e, 4803)
    out = run_bwd(e, dO, dS)
    assert torch.equal(out[5].cpu(), dS)


def test_gdn_bwd_long_segment_sampled():
    """8192 tokens (128 chunks, several superchunks) over 8 heads; the oracle
    runs two of them."""
    B, L, H, D = 1, 8192, 8, 128
    say(f"[gdn bwd] long segment L={L} H={H}")
    inp = synth.make_gdn_inputs(B, L, H, D, seed=4900)
    dO, dS = grads_inputs(inp, 4901)
    got = run_bwd(inp, dO, dS)
    heads = [1, 6]
    want = ref_bwd(inp, dO, dS, heads)
    sub = [x[:, :, heads] for x in got[:5]] + [got[5][:, heads]]
    check_bwd(sub, want)


def test_gdn_bwd_chained_segments():
    """Forward chained through S, backward chained through dS in reverse: the
    gradients of the concatenated segments equal the oracle's over the whole
    sequence."""
    B, H, D = 1, 2, 128
    segs = [256, 64, 320]
    say(f"[gdn bwd] chained {segs}")
    inp = synth.make_gdn_inputs(B, sum(segs), H, D, seed=5000)
    dO, dS_out = grads_inputs(inp, 5001)
    g = {k: (v.to(DEV) if isinstance(v, torch.Tensor) else v) for k, v in inp.items()}
    dOd, dSd = dO.to(DEV), dS_out.to(DEV)
    starts = [sum(segs[:i]) for i in range(len(segs))]
    sl = lambda x, t, n: x[:, t:t + n]
    S, bounds = g["S_in"], []
    for t, n in zip(starts, segs):
        bounds.append(S)
        _, S = sf.gdn_fwd(sl(g["q"], t, n), sl(g["k"], t, n), sl(g["v"], t, n), sl(g["g"], t, n),
                          sl(g["beta"], t, n), S)
    dS, parts = dSd, []
    for t, n, S0 in reversed(list(zip(starts, segs, bounds))):
        out = sf.gdn_bwd(sl(g["q"], t, n), sl(g["k"], t, n), sl(g["v"], t, n), sl(g["g"], t, n),
                         sl(g["beta"], t, n), S0, sl(dOd, t, n), dS)
        parts.insert(0, out[:5])
        dS = out[5]
    torch.cuda.synchronize()
    got = [torch.cat([p[i] for p in parts], 1) for i in range(5)] + [dS]
    check_bwd(got, ref_bwd(inp, dO, dS_out))


def test_gdn_head_major_layout():
    """q, k, v, dO stored head-major ([B, H, L, D] in memory) and g, beta as
    [B, H, L], passed as [B, L, H, ...] views: the strides go through the ABI
    and the results match the oracle (forward and backward)."""
    B, L, H, D = 2, 320, 3, 128
    say(f"[gdn] head-major layout B={B} L={L} H={H}")
    inp = synth.make_gdn_inputs(B, L, H, D, seed=5100)
    dO, dS_out = grads_inputs(inp, 5101)

    def hm(x):  # same values, head-major memory
        p = (0, 2, 1, 3) if x.dim() == 4 else (0, 2, 1)
        return x.permute(*p).contiguous().permute(*p).to(DEV)

    q, k, v, g, beta = (hm(inp[n]) for n in ("q", "k", "v", "g", "beta"))
    do = hm(dO)
    assert q.stride(1) == D and q.stride(2) == L * D and g.stride(1) == 1
    S_in = inp["S_in"].to(DEV)
    o, S = sf.gdn_fwd(q, k, v, g, beta, S_in)
    grads = sf.gdn_bwd(q, k, v, g, beta, S_in, do, dS_out.to(DEV))
    torch.cuda.synchronize()
    assert o.stride() == q.stride() and grads[3].stride() == g.stride()
    ro, rS = ref(inp)
    assert_close("o", o, ro, "bf16")
    assert_close("S_out", S, rS, "bf16")
    check_bwd(grads, ref_bwd(inp, dO, dS_out))


def test_gdn_full_size_segment_sampled():
    """The largest segment of the 256K-context workload at full size
    (B 1, L 65536, H 40, d 128, the library's own superchunk choice): forward
    and backward on the GPU, two heads against the oracle."""
    B, L, H, D = 1, 65536, 40, 128
    say(f"[gdn] full-size segment L={L} H={H}")
    inp = synth.make_gdn_inputs(B, L, H, D, device=DEV, seed=5200)
    gen = torch.Generator(device=DEV).manual_seed(5201)
    dO = torch.randn((B, L, H, D), device=DEV, generator=gen).to(torch.bfloat16)
    dS_out = 0.1 * torch.randn((B, H, D, D), device=DEV, generator=gen)
    o, S = sf.gdn_fwd(inp["q"], inp["k"], inp["v"], inp["g"], inp["beta"], inp["S_in"])
    grads = sf.gdn_bwd(inp["q"], inp["k"], inp["v"], inp["g"], inp["beta"], inp["S_in"], dO, dS_out)
    torch.cuda.synchronize()
    heads = [0, 37]
    cpu = {k: v[:, :, heads].cpu() for k, v in inp.items() if k != "S_in"}
    cpu["S_in"] = inp["S_in"][:, heads].cpu()
    ro, rS = ref(cpu)
    assert_close("o", o[:, :, heads], ro, "bf16")
    assert_close("S_out", S[:, heads], rS, "bf16")
    sub = [x[:, :, heads] for x in grads[:5]] + [grads[5][:, heads]]
    check_bwd(sub, ref_bwd(cpu, dO[:, :, heads].cpu(), dS_out[:, heads].cpu()))


@pytest.mark.parametrize("D,ts", [(128, 0), (128, 128), (64, 0)])
def test_gdn_chain_entry_points(D, ts):
    """sf_gdn_chain_fwd / sf_gdn_chain_bwd over nonuniform segments (one of
    them a single superchunk when ts = 128): forward, V^new and every gradient
    against the oracle over the whole sequence; the scans overlapped on an aux
    stream give bitwise the same results as serialised on one stream, and the
    backward that reads the forward's kept superchunk states and maps gives
    bitwise the results of the one that replays them."""
    B, H = 1, 3
    segs = [256, 64, 384, 192]
    say(f"[gdn chain] D={D} segs={segs} ts={ts}")
    inp = synth.make_gdn_inputs(B, sum(segs), H, D, seed=5300 + ts + D)
    dO, dS_final = grads_inputs(inp, 5301 + ts + D)
    g = {k: (v.to(DEV) if isinstance(v, torch.Tensor) else v) for k, v in inp.items()}
    args = (g["q"], g["k"], g["v"], g["g"], g["beta"], segs)
    res = {}
    for ov in (True, False):
        for keep in (False, True):
            out = sf.gdn_chain_fwd(*args, g["S_in"], ts=ts, overlap=ov, with_v_new=True, keep_states=keep)
            o, S_bnd, vn = out[:3]
            grads = sf.gdn_chain_bwd(*args, S_bnd, dO.to(DEV), dS_final.to(DEV), ts=ts, overlap=ov,
                                     ckpt=out[3] if keep else None)
            torch.cuda.synchronize()
            res[ov, keep] = (o, S_bnd, vn) + tuple(grads)
    for key in res:
        for x, y in zip(res[True, False], res[key]):
            assert torch.equal(x, y), key
    res[True] = res[True, False]
    o, S_bnd, vn = res[True][:3]
    ro, rS, ru = gdn.forward(*(to64(inp[x]) for x in ("q", "k", "v", "g", "beta", "S_in")), threads=cores(),
                             with_u=True)
    assert_close("o", o, ro, "bf16")
    assert_close("v_new", vn, ru, "bf16")
    assert_close("S_out", S_bnd[-1], rS, "bf16")
    t = 0
    for i, n in enumerate(segs[:-1]):  # interior boundary states
        t += n
        _, Si = gdn.forward(*(to64(inp[x][:, :t]) for x in ("q", "k", "v", "g", "beta")), to64(inp["S_in"]),
                            threads=cores())
        assert_close(f"S_bnd{i + 1}", S_bnd[i + 1], Si, "bf16")
    check_bwd(res[True][3:], ref_bwd(inp, dO, dS_final))
