"""GPU parity of attention over key segments and of the (O, LSE) merge: the
HIP path (through the C ABI) against the oracle, element by element.

Queries and keys of different lengths, per-segment forwards merged on the GPU
against the full attention, per-segment backwards with the merged statistics
(dQ accumulated across segments) against the full backward, and the merge
kernel alone on random partials (including a NaN row)."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_util import TOL_LSE_MAX, assert_close, rel_l2, to_device, torch

pytestmark = pytest.mark.gpu


def np64(t):
    return t.detach().double().cpu().numpy()


def cross_inputs(B, H, Nq, Nk, d, seed):
    """q, dout with Nq rows and k, v with Nk rows (seeded, like every input)."""
    xq = workloads.make_small_inputs(B, H, Nq, d, seed=seed, with_dout=True)
    xk = workloads.make_small_inputs(B, H, Nk, d, seed=seed + 7919, with_dout=False)
    return {"q": xq["q"], "dout": xq["dout"], "k": xk["k"], "v": xk["v"]}


CROSS = [(1, 2, 300, 77, 64), (2, 1, 129, 500, 128), (1, 1, 1, 1, 128), (1, 1, 64, 1, 64), (1, 1, 3, 4097, 128),
         (1, 2, 1000, 33, 128)]


@pytest.mark.parametrize("B,H,Nq,Nk,d", CROSS)
def test_fwd_kv_cross_lengths(B, H, Nq, Nk, d):
    import paper_2405_15780_amd as va

    print(f"case B={B} H={H} Nq={Nq} Nk={Nk} d={d}", flush=True)
    x = cross_inputs(B, H, Nq, Nk, d, seed=300 + Nq + Nk + d)
    scale = 1.0 / np.sqrt(d)
    o, lse = va.fwd(to_device(x["q"]), to_device(x["k"]), to_device(x["v"]), scale)
    torch().cuda.synchronize()
    ref_o, ref_lse = oracle.forward(x["q"], x["k"], x["v"], scale)
    assert_close({"o": np64(o), "lse": np64(lse)}, {"o": ref_o, "lse": ref_lse}, names=("o", "lse"),
                 label=f"fwd_kv {B},{H},{Nq},{Nk},{d}")


SEGMENTS = [(64, 700, (131, 450)), (128, 700, (131, 450)), (128, 2100, (1, 64, 1000, 2047)), (64, 95, (94,))]


def _segments(N, cuts):
    edges = [0] + list(cuts) + [N]
    return list(zip(edges[:-1], edges[1:]))


@pytest.mark.parametrize("d,N,cuts", SEGMENTS)
def test_segment_forwards_merged_equal_full_attention(d, N, cuts):
    import paper_2405_15780_amd as va

    t = torch()
    print(f"case d={d} N={N} cuts={cuts}", flush=True)
    x = workloads.make_small_inputs(1, 2, N, d, seed=400 + N + d, with_dout=False)
    scale = 1.0 / np.sqrt(d)
    q = to_device(x["q"])
    parts = []
    for a, b in _segments(N, cuts):
        k = to_device(np.ascontiguousarray(x["k"][:, :, a:b]))
        v = to_device(np.ascontiguousarray(x["v"][:, :, a:b]))
        parts.append(va.fwd(q, k, v, scale))
    o_parts = t.stack([p[0] for p in parts]).contiguous()
    lse_parts = t.stack([p[1] for p in parts]).contiguous()
    o, lse = va.merge(o_parts, lse_parts)
    o_full, lse_full = va.fwd(q, to_device(x["k"]), to_device(x["v"]), scale)
    t.cuda.synchronize()
    ref_o, ref_lse = oracle.forward(x["q"], x["k"], x["v"], scale)
    assert_close({"o": np64(o), "lse": np64(lse)}, {"o": ref_o, "lse": ref_lse}, names=("o", "lse"),
                 label=f"merged segments d={d} N={N}")
    # the merge of the GPU partials agrees with the GPU's own full forward far
    # inside the oracle tolerance (both are fp32 sums of the same bf16 terms)
    assert float(np.abs(np64(o) - np64(o_full)).max()) <= 2e-3
    assert float(np.abs(np64(lse) - np64(lse_full)).max()) <= 1e-4


@pytest.mark.parametrize("d,N,cuts", SEGMENTS[:3])
def test_segment_backwards_with_merged_statistics_equal_full_backward(d, N, cuts):
    import paper_2405_15780_amd as va

    t = torch()
    print(f"case d={d} N={N} cuts={cuts}", flush=True)
    x = workloads.make_small_inputs(1, 2, N, d, seed=500 + N + d, with_dout=True)
    scale = 1.0 / np.sqrt(d)
    q, dout = to_device(x["q"]), to_device(x["dout"])
    o, lse = va.fwd(q, to_device(x["k"]), to_device(x["v"]), scale)
    dq = t.zeros((1, 2, N, d), dtype=t.float32, device="cuda")
    dk_parts, dv_parts = [], []
    for a, b in _segments(N, cuts):
        k = to_device(np.ascontiguousarray(x["k"][:, :, a:b]))
        v = to_device(np.ascontiguousarray(x["v"][:, :, a:b]))
        dk = t.empty((1, 2, b - a, d), dtype=t.float32, device="cuda")
        dv = t.empty_like(dk)
        va.bwd(q, k, v, o, lse, dout, scale, out=(dq, dk, dv), accumulate_dq=True)
        dk_parts.append(dk)
        dv_parts.append(dv)
    t.cuda.synchronize()
    got = {"dq": np64(dq), "dk": np64(t.cat(dk_parts, dim=2)), "dv": np64(t.cat(dv_parts, dim=2))}
    ref = oracle.forward_backward(x["q"], x["k"], x["v"], x["dout"], scale)
    assert_close(got, ref, names=("dq", "dk", "dv"), label=f"segment backward d={d} N={N}")


def test_dq_overwrite_ignores_previous_contents():
    # without the accumulate flag dq is written, not added to
    import paper_2405_15780_amd as va

    t = torch()
    x = cross_inputs(1, 1, 100, 60, 64, seed=611)
    scale = 0.125
    q, k, v, dout = (to_device(x[n]) for n in ("q", "k", "v", "dout"))
    o, lse = va.fwd(q, k, v, scale)
    dq = t.full((1, 1, 100, 64), 123.0, dtype=t.float32, device="cuda")
    dk = t.empty((1, 1, 60, 64), dtype=t.float32, device="cuda")
    dv = t.empty_like(dk)
    va.bwd(q, k, v, o, lse, dout, scale, out=(dq, dk, dv))
    t.cuda.synchronize()
    fwd_o, fwd_lse = oracle.forward(x["q"], x["k"], x["v"], scale)
    dq_ref, dk_ref, dv_ref = oracle.segment_backward(x["q"], x["k"], x["v"], x["dout"], fwd_o, fwd_lse, scale)
    assert rel_l2(np64(dq), dq_ref) <= 1e-2
    assert rel_l2(np64(dk), dk_ref) <= 1e-2
    assert rel_l2(np64(dv), dv_ref) <= 1e-2


@pytest.mark.parametrize("d", [8, 64, 72, 128, 136, 160])
def test_merge_kernel_against_oracle(d):
    import paper_2405_15780_amd as va

    t = torch()
    rng = np.random.default_rng(700 + d)
    P, B, H, N = 3, 2, 2, 77
    o_parts = rng.standard_normal((P, B, H, N, d)).astype(np.float32)
    lse_parts = (20.0 * rng.standard_normal((P, B, H, N))).astype(np.float32)
    lse_parts[1, 1, 0, 5] = np.nan  # poisons that row only
    o, lse = va.merge(t.from_numpy(o_parts).cuda(), t.from_numpy(lse_parts).cuda())
    t.cuda.synchronize()
    ref_o, ref_lse = oracle.merge(o_parts, lse_parts)
    got_o, got_lse = np64(o), np64(lse)
    nan_rows = np.isnan(ref_lse)
    assert nan_rows.sum() == 1 and np.isnan(got_lse[nan_rows]).all() and np.isnan(got_o[nan_rows]).all()
    ok = ~nan_rows
    assert float(np.abs(got_lse[ok] - ref_lse[ok]).max()) <= 1e-5 * max(1.0, float(np.abs(ref_lse[ok]).max()))
    assert float(np.abs(got_o[ok] - ref_o[ok]).max()) <= 1e-5
    assert float(np.abs(got_lse[ok] - ref_lse[ok]).max()) <= TOL_LSE_MAX
