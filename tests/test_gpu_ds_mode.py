"""GPU parity of the dS mode of the backward pass (VITATTN_BWD_STORE_DS): the
dK/dV kernel stores its bf16 dS blocks and dQ is computed from them instead
of recomputing S and dP. dQ, dK and dV are compared with the oracle element by
element (several tiles, ragged tails, the tile widths of the other head dims,
sequence-major operands, key segments with dQ accumulation); dK and dV must
be bitwise equal to the default mode (the same kernel arithmetic; only the
dS stores are added)."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_util import assert_close, to_device, torch

pytestmark = pytest.mark.gpu


def np64(t):
    return t.detach().double().cpu().numpy()


def both_modes(x, scale):
    import paper_2405_15780_amd as va

    dev = {n: to_device(a) for n, a in x.items()}
    o, lse = va.fwd(dev["q"], dev["k"], dev["v"], scale)
    ref_mode = va.bwd(dev["q"], dev["k"], dev["v"], o, lse, dev["dout"], scale)
    ds_mode = va.bwd(dev["q"], dev["k"], dev["v"], o, lse, dev["dout"], scale, store_ds=True)
    torch().cuda.synchronize()
    return o, lse, ref_mode, ds_mode


SHAPES = [(1, 2, 300, 64), (2, 1, 129, 128), (1, 1, 1, 64), (1, 1, 64, 128), (1, 1, 1000, 72), (1, 1, 700, 160),
          (1, 2, 4097, 128), (2, 3, 200, 40)]


@pytest.mark.parametrize("B,H,N,d", SHAPES)
def test_ds_mode_full_compare(B, H, N, d):
    t = torch()
    print(f"case dS mode B={B} H={H} N={N} d={d}", flush=True)
    x = workloads.make_small_inputs(B, H, N, d, seed=4400 + N + d)
    scale = 1.0 / np.sqrt(d)
    o, lse, (dq0, dk0, dv0), (dq, dk, dv) = both_modes(x, scale)
    assert t.equal(dk, dk0) and t.equal(dv, dv0), "dK / dV differ from the default mode"
    ref = oracle.forward_backward(x["q"], x["k"], x["v"], x["dout"], scale)
    assert_close({"dq": np64(dq), "dk": np64(dk), "dv": np64(dv)}, ref, names=("dq", "dk", "dv"),
                 label=f"dS mode {B},{H},{N},{d}")
    # the two modes' dQ differ only by the rounding of dS to bf16
    rel = float(t.linalg.norm(dq - dq0) / t.linalg.norm(dq0)) if N > 1 else float((dq - dq0).abs().max())
    assert rel < 5e-3, rel


def test_ds_mode_16k_tokens_head_compare():
    print("case dS mode N=16384 d=128", flush=True)
    B, H, N, d = 1, 2, 16384, 128
    x = workloads.make_small_inputs(B, H, N, d, seed=4900)
    scale = 1.0 / np.sqrt(d)
    _, _, _, (dq, dk, dv) = both_modes(x, scale)
    ref = oracle.forward_backward(x["q"], x["k"], x["v"], x["dout"], scale, heads=[(0, 1)])
    got = {"dq": np64(dq[0, 1]), "dk": np64(dk[0, 1]), "dv": np64(dv[0, 1])}
    assert_close(got, {n: ref[n][0, 1] for n in ("dq", "dk", "dv")}, names=("dq", "dk", "dv"),
                 label="dS mode N=16384 head (0,1)")


@pytest.mark.parametrize("d", [64, 160])
def test_ds_mode_sequence_major_segments_accumulate(d):
    """Key segments of a sequence-major layout, dQ summed over the segments."""
    import paper_2405_15780_amd as va

    t = torch()
    B, H, Nq, N = 1, 2, 150, 330
    cuts = [(0, 97), (97, 330)]
    print(f"case dS mode strided segments d={d}", flush=True)
    xq = workloads.make_small_inputs(B, H, Nq, d, seed=5100 + d)
    xk = workloads.make_small_inputs(B, H, N, d, seed=5200 + d, with_dout=False)
    scale = 1.0 / np.sqrt(d)

    def bnhd(bits):
        return to_device(np.ascontiguousarray(bits.transpose(0, 2, 1, 3))).transpose(1, 2)

    def bnhd_out(n):
        return t.empty((B, n, H, d), dtype=t.float32, device="cuda").transpose(1, 2)

    ref_o, ref_lse = oracle.forward(xq["q"], xk["k"], xk["v"], scale)
    ref_dq, ref_dk, ref_dv = oracle.segment_backward(xq["q"], xk["k"], xk["v"], xq["dout"], ref_o, ref_lse, scale)
    qs, gs = bnhd(xq["q"]), bnhd(xq["dout"])
    o, lse = va.fwd(qs, bnhd(xk["k"]), bnhd(xk["v"]), scale)
    dq = bnhd_out(Nq).zero_()
    for a, b in cuts:
        dk, dv = bnhd_out(b - a), bnhd_out(b - a)
        va.bwd(qs, bnhd(xk["k"][:, :, a:b]), bnhd(xk["v"][:, :, a:b]), o, lse, gs, scale, out=(dq, dk, dv),
               accumulate_dq=True, store_ds=True)
        t.cuda.synchronize()
        assert_close({"dk": np64(dk), "dv": np64(dv)}, {"dk": ref_dk[:, :, a:b], "dv": ref_dv[:, :, a:b]},
                     names=("dk", "dv"), label=f"dS mode segment {a}:{b} d={d}")
    assert_close({"dq": np64(dq)}, {"dq": ref_dq}, names=("dq",), label=f"dS mode segments dQ d={d}")


def test_ds_mode_stage_entry_points_match_the_whole_call():
    import paper_2405_15780_amd as va

    t = torch()
    print("case dS mode stages", flush=True)
    B, H, N, d = 1, 2, 777, 128
    x = workloads.make_small_inputs(B, H, N, d, seed=5300)
    scale = 1.0 / np.sqrt(d)
    dev = {n: to_device(a) for n, a in x.items()}
    o, lse = va.fwd(dev["q"], dev["k"], dev["v"], scale)
    dq, dk, dv = va.bwd(dev["q"], dev["k"], dev["v"], o, lse, dev["dout"], scale, store_ds=True)
    ws = t.empty(va.workspace_bytes_kv(B, H, N, N, d, va.VITATTN_BWD_STORE_DS) // 4, device="cuda")
    dq2, dk2, dv2 = (t.empty_like(dq) for _ in range(3))
    va.bwd_rowdot(o, dev["dout"], lse, ws)
    va.bwd_dkdv_ds(dev["q"], dev["k"], dev["v"], dev["dout"], lse, dk2, dv2, ws, scale)
    va.bwd_dq_from_ds(dev["k"], dq2, ws, scale)
    t.cuda.synchronize()
    assert t.equal(dq, dq2) and t.equal(dk, dk2) and t.equal(dv, dv2)
