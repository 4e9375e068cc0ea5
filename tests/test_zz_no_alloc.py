"""The allocation-free segment forward (sf_segment_fwd_noalloc, through the C
ABI) against sf_segment_fwd with the same tuning: bitwise equal outputs on two
calls in a row, the second on a smaller input (the scratch keeps the first
call's contents), both against the oracle too; shapes whose workspace exceeds
the static scratch are rejected before any launch."""
import ctypes

import pytest
import torch

import paper_2608_06838_amd as sf
from paper_2608_06838_amd import _lib, synth
from tests._helpers import assert_close, oracle_run

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _case(B, H, L, ts, seed):
    w = synth.workload("mid_bf16", B=B, H=H, D=128, s_in_std=0.1)
    inp = synth.make_inputs(w, device="cpu", seed=seed, L=L)
    g = {k: (v.to(DEV) if isinstance(v, torch.Tensor) else v) for k, v in inp.items()}
    need = sf.fwd_workspace_bytes(g["q"], g["g"], ts=ts)
    assert 0 < need <= _lib.NOALLOC_SCRATCH_BYTES  # the scratch is used
    print(f"[noalloc] B={B} H={H} L={L} ts={ts} scratch bytes used {need}", flush=True)
    o_ref, S_ref = sf.segment_fwd(g["q"], g["k"], g["v"], g["g"], g["S_in"], ts=ts)
    o = torch.empty_like(g["q"])
    S = torch.empty((B, H, 128, 128), dtype=torch.float32, device=DEV)
    sf.segment_fwd_noalloc(g["q"], g["k"], g["v"], g["g"], g["S_in"], o, S, ts=ts)
    torch.cuda.synchronize()
    return inp, (o_ref, S_ref), (o, S)


def test_noalloc_matches_segment_fwd():
    big = _case(1, 4, 2048, 256, seed=71)      # 8 superchunks of 256 tokens
    small = _case(1, 2, 1024, 192, seed=72)    # then fewer, ragged ones
    for inp, ref, got in (big, small):
        assert torch.equal(got[0], ref[0]) and torch.equal(got[1], ref[1])
        r = oracle_run(inp)
        assert_close("o", got[0], r["o"], "bf16")
        assert_close("S_out", got[1], r["S_out"], "bf16")


def test_noalloc_rejects_oversized_shape():
    sh = _lib.SfShape()
    sh.B, sh.H, sh.Dk, sh.Dv, sh.L, sh.chunk, sh.io_dtype, sh.gate = 1, 40, 128, 128, 65536, 64, _lib.SF_BF16, 0
    t = _lib.SfTuning()
    t.ts = 64  # 1024 superchunks: 2.7 GB of states
    p = [ctypes.c_void_p(0x7F0000000000 + i * (1 << 34)) for i in range(6)]
    rc = _lib.lib().sf_segment_fwd_noalloc(ctypes.byref(sh), p[0], p[1], p[2], p[3], None, p[4], p[5],
                                           ctypes.byref(t), None)
    assert rc == _lib.SF_E_WORKSPACE
    assert b"allocation-free" in _lib.lib().sf_last_error()
