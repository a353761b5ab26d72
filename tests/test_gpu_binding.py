"""The Python binding rejects device tensors whose dtype, shape, layout or
device does not match what the C ABI will index (a mismatch would otherwise
be an out-of-bounds access on the GPU). Every case raises before any launch."""
import pytest

from gpu_util import torch

pytestmark = pytest.mark.gpu

B, H, N, d = 1, 2, 40, 64


def dev(*shape, dtype=None):
    t = torch()
    return t.zeros(shape, dtype=dtype or t.float32, device="cuda")


def operands():
    t = torch()
    q, k, v, g = (dev(B, H, N, d, dtype=t.bfloat16) for _ in range(4))
    return q, k, v, g


def test_fwd_and_bwd_reject_mismatched_outputs_and_inputs():
    import paper_2405_15780_amd as va

    t = torch()
    print("case binding fwd/bwd", flush=True)
    q, k, v, g = operands()
    o, lse = va.fwd(q, k, v)
    t.cuda.synchronize()
    with pytest.raises(TypeError):
        va.fwd(q, k, v, out=(dev(B, H, N - 1, d), lse))  # o one row short
    with pytest.raises(TypeError):
        va.fwd(q, k, v, out=(o, dev(B, H, N, dtype=t.bfloat16)))  # lse of the wrong dtype
    with pytest.raises(TypeError):
        va.fwd(q, k, v, out=(o, dev(B, H, 2 * N)[..., ::2]))  # lse not contiguous
    with pytest.raises(TypeError):
        va.bwd(q, k, v, o.to(t.bfloat16), lse, g)  # o must be fp32
    with pytest.raises(TypeError):
        va.bwd(q, k, v, o, lse[..., :-1], g)  # lse one row short
    with pytest.raises(TypeError):
        va.bwd(q, k, v, o, lse, g[:, :, :-1])  # dout one row short
    dq = dev(B, H, N, d)
    with pytest.raises(TypeError):
        va.bwd(q, k, v, o, lse, g, out=(dq, dev(B, H, N, d // 2), dev(B, H, N, d)))
    with pytest.raises(TypeError):
        va.bwd(q, k, v, o, lse, g, workspace=dev(1).expand(1 << 20))  # a workspace of one float
    # strided outputs with d contiguous are accepted; d-strided ones are not
    wide = dev(B, H, N, 2 * d)
    va.fwd(q, k, v, out=(wide[..., :d], lse))
    with pytest.raises(TypeError):
        va.fwd(q, k, v, out=(wide[..., ::2], lse))
    t.cuda.synchronize()


def test_stage_entry_points_reject_mismatches():
    import paper_2405_15780_amd as va

    t = torch()
    print("case binding stages", flush=True)
    q, k, v, g = operands()
    o, lse = va.fwd(q, k, v)
    ws = dev(va.workspace_bytes(B, H, N, d) // 4 + 64)
    dk, dv = dev(B, H, N, d), dev(B, H, N, d)
    with pytest.raises(TypeError):
        va.bwd_rowdot(o, g, lse, ws[::2])  # strided workspace
    with pytest.raises(TypeError):
        va.bwd_dkdv(q, k, v, g, lse, dk.to(t.bfloat16), dv, ws)  # dk must be fp32
    with pytest.raises(TypeError):
        va.bwd_dkdv(q, k[:, :, :-1], v, g, lse, dk, dv, ws)  # k one row short
    with pytest.raises(TypeError):
        va.bwd_dq(q, k, v, g, lse, dev(B, H, N, d + 8), ws)
    with pytest.raises(TypeError):
        va.bwd_dq_from_ds(k, dev(B, H, N, d).transpose(1, 2), ws)  # dq not contiguous
    t.cuda.synchronize()


def test_merge_and_aggregation_reject_mismatches():
    import paper_2405_15780_amd as va

    t = torch()
    print("case binding merge/agg", flush=True)
    parts, lse_parts = dev(3, B, H, N, d), dev(3, B, H, N)
    with pytest.raises(TypeError):
        va.merge(parts, lse_parts, out=(dev(B, H, N, d), dev(B, H, N - 1)))
    with pytest.raises(TypeError):
        va.merge(parts, lse_parts[:2])
    M, C = 3, 5
    qa = dev(H, d, dtype=t.bfloat16)
    ka, va_ = dev(M, H, C, d, dtype=t.bfloat16), dev(M, H, C, d, dtype=t.bfloat16)
    oa, la = va.agg_fwd(qa, ka, va_)
    ga = dev(M, H, d, dtype=t.bfloat16)
    with pytest.raises(TypeError):
        va.agg_bwd(qa, ka, va_, oa, la[:, :1], ga)  # lse [M, 1] instead of [M, H]
    with pytest.raises(TypeError):
        va.agg_bwd(qa, ka, va_, oa.to(t.bfloat16), la, ga)
    t.cuda.synchronize()
