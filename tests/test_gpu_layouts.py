"""GPU parity of head-dim and layout generality: head dims other than 64 and
128 (the paper's d = 72 of ViT-10B, Table I, and d = 160 of the Sec. V-C
model, plus every tile width's boundary cases), and operands in other
layouts (the sequence-major [B, N, H, d] an all-to-all produces, rows padded
to a larger pitch, keys and values shared by several heads). The HIP path is
compared element by element with the oracle on the logical [B, H, N, d]
arrays, and layouts are also compared bitwise with the dense call on the same
values (the kernels are the same; only addresses differ)."""
import numpy as np
import pytest

import oracle
import workloads
from gpu_util import assert_close, to_device, torch

pytestmark = pytest.mark.gpu


def np64(t):
    return t.detach().double().cpu().numpy()


def run(q, k, v, dout, scale, outs=None):
    """Forward and backward through the binding on device tensors of any
    layout; outs = (o, lse, dq, dk, dv) preallocated views, or None."""
    import paper_2405_15780_amd as va

    o, lse = va.fwd(q, k, v, scale, out=None if outs is None else outs[:2])
    dq, dk, dv = va.bwd(q, k, v, o, lse, dout, scale, out=None if outs is None else outs[2:])
    torch().cuda.synchronize()
    return {"o": o, "lse": lse, "dq": dq, "dk": dk, "dv": dv}


def dense_run(x, scale):
    return run(*(to_device(x[n]) for n in ("q", "k", "v", "dout")), scale)


# every tile width, with the 96-wide tile on both sides of its contraction
# boundary (d <= 80 contracts over five 16-column steps, 88 and 96 over six)
HEAD_DIMS = [8, 24, 40, 72, 80, 88, 96, 104, 136, 160]


@pytest.mark.parametrize("d", HEAD_DIMS)
@pytest.mark.parametrize("B,H,N", [(1, 2, 300), (2, 1, 129)])
def test_head_dims_full_compare(B, H, N, d):
    print(f"case B={B} H={H} N={N} d={d}", flush=True)
    x = workloads.make_small_inputs(B, H, N, d, seed=500 + N + d)
    scale = 1.0 / np.sqrt(d)
    got = {n: np64(t) for n, t in dense_run(x, scale).items()}
    ref = oracle.forward_backward(x["q"], x["k"], x["v"], x["dout"], scale)
    assert_close(got, ref, label=f"head dim {B},{H},{N},{d}")


@pytest.mark.parametrize("d,N", [(72, 1), (160, 1), (72, 1000), (160, 1000), (72, 4097), (160, 2049)])
def test_paper_head_dims_edges_and_tiles(d, N):
    print(f"case N={N} d={d}", flush=True)
    x = workloads.make_small_inputs(1, 1, N, d, seed=900 + N + d)
    scale = 1.0 / np.sqrt(d)
    got = {n: np64(t) for n, t in dense_run(x, scale).items()}
    ref = oracle.forward_backward(x["q"], x["k"], x["v"], x["dout"], scale)
    assert_close(got, ref, label=f"paper head dim N={N} d={d}")


def _bnhd(bits):
    """Device bf16 tensor stored sequence-major [B, N, H, d], returned as its
    [B, H, N, d] view."""
    return to_device(np.ascontiguousarray(bits.transpose(0, 2, 1, 3))).transpose(1, 2)


def _bnhd_out(B, H, N, d):
    t = torch()
    return t.empty((B, N, H, d), dtype=t.float32, device="cuda").transpose(1, 2)


@pytest.mark.parametrize("d", [64, 72, 128, 160])
def test_sequence_major_layout(d):
    t = torch()
    B, H, N = 2, 3, 257
    print(f"case [B,N,H,d] d={d}", flush=True)
    x = workloads.make_small_inputs(B, H, N, d, seed=1300 + d)
    scale = 1.0 / np.sqrt(d)
    ins = [_bnhd(x[n]) for n in ("q", "k", "v", "dout")]
    assert not ins[0].is_contiguous() and ins[0].stride() == (N * H * d, d, H * d, 1)
    outs = (_bnhd_out(B, H, N, d), t.empty((B, H, N), dtype=t.float32, device="cuda"),
            *(_bnhd_out(B, H, N, d) for _ in range(3)))
    res = run(*ins, scale, outs=outs)
    ref = oracle.forward_backward(x["q"], x["k"], x["v"], x["dout"], scale)
    assert_close({n: np64(v) for n, v in res.items()}, ref, label=f"[B,N,H,d] d={d}")
    dense = dense_run(x, scale)
    for n in res:
        assert t.equal(res[n], dense[n]), f"{n} differs bitwise from the dense layout"


@pytest.mark.parametrize("d,pad_in,pad_out", [(64, 8, 4), (72, 24, 8), (128, 64, 12), (160, 8, 4)])
def test_padded_rows_leave_padding_untouched(d, pad_in, pad_out):
    t = torch()
    B, H, N = 1, 2, 200
    print(f"case padded rows d={d} pad_in={pad_in} pad_out={pad_out}", flush=True)
    x = workloads.make_small_inputs(B, H, N, d, seed=1700 + d)
    scale = 1.0 / np.sqrt(d)

    def padded_in(bits):
        buf = t.zeros((B, H, N, d + pad_in), dtype=t.bfloat16, device="cuda")
        buf[..., :d] = to_device(bits)
        return buf, buf[..., :d]

    sentinel = 12345.0
    out_bufs = [t.full((B, H, N, d + pad_out), sentinel, dtype=t.float32, device="cuda") for _ in range(4)]
    outs = (out_bufs[0][..., :d], t.empty((B, H, N), dtype=t.float32, device="cuda"),
            *(b[..., :d] for b in out_bufs[1:]))
    ins = [padded_in(x[n])[1] for n in ("q", "k", "v", "dout")]
    res = run(*ins, scale, outs=outs)
    dense = dense_run(x, scale)
    for n in res:
        assert t.equal(res[n], dense[n]), f"{n} differs bitwise from the dense layout"
    for b in out_bufs:
        assert bool((b[..., d:] == sentinel).all()), "a write landed in the row padding"
    ref = oracle.forward_backward(x["q"], x["k"], x["v"], x["dout"], scale)
    assert_close({n: np64(v) for n, v in res.items()}, ref, label=f"padded d={d}")


@pytest.mark.parametrize("d", [64, 72])
def test_keys_shared_by_heads(d):
    """K and V with head stride 0 (one key head serving H query heads)."""
    t = torch()
    B, H, N = 2, 4, 300
    print(f"case shared K/V heads d={d}", flush=True)
    x = workloads.make_small_inputs(B, H, N, d, seed=2100 + d)
    k1, v1 = x["k"][:, :1], x["v"][:, :1]
    kx = to_device(k1).expand(B, H, N, d)
    vx = to_device(v1).expand(B, H, N, d)
    assert kx.stride(1) == 0
    scale = 1.0 / np.sqrt(d)
    res = run(to_device(x["q"]), kx, vx, to_device(x["dout"]), scale)
    kb = np.broadcast_to(k1, (B, H, N, d)).copy()
    vb = np.broadcast_to(v1, (B, H, N, d)).copy()
    ref = oracle.forward_backward(x["q"], kb, vb, x["dout"], scale)
    assert_close({n: np64(v) for n, v in res.items()}, ref, label=f"shared K/V d={d}")


@pytest.mark.parametrize("d", [72, 160])
def test_sequence_major_key_segments_accumulate_dq(d):
    """Nq != Nk key segments in [B, N, H, d], dQ summed over segments, equal
    bitwise to the same calls on dense operands."""
    import paper_2405_15780_amd as va

    t = torch()
    B, H, Nq, N = 1, 2, 150, 330
    cuts = [(0, 97), (97, 330)]
    print(f"case strided segments d={d}", flush=True)
    xq = workloads.make_small_inputs(B, H, Nq, d, seed=2500 + d)
    xk = workloads.make_small_inputs(B, H, N, d, seed=2600 + d, with_dout=False)
    scale = 1.0 / np.sqrt(d)
    ref_o, ref_lse = oracle.forward(xq["q"], xk["k"], xk["v"], scale)
    ref_dq, ref_dk, ref_dv = oracle.segment_backward(xq["q"], xk["k"], xk["v"], xq["dout"], ref_o, ref_lse, scale)
    ref = {"o": ref_o, "lse": ref_lse, "dq": ref_dq, "dk": ref_dk, "dv": ref_dv}
    o, lse = va.fwd(_bnhd(xq["q"]), _bnhd(xk["k"]), _bnhd(xk["v"]), scale)
    q_s, g_s = _bnhd(xq["q"]), _bnhd(xq["dout"])
    q_d, g_d = to_device(xq["q"]), to_device(xq["dout"])
    dq_s = _bnhd_out(B, H, Nq, d).zero_()
    dq_d = t.zeros((B, H, Nq, d), dtype=t.float32, device="cuda")
    for a, b in cuts:
        ks, vs = _bnhd(xk["k"][:, :, a:b]), _bnhd(xk["v"][:, :, a:b])
        dk_s, dv_s = _bnhd_out(B, H, b - a, d), _bnhd_out(B, H, b - a, d)
        va.bwd(q_s, ks, vs, o, lse, g_s, scale, out=(dq_s, dk_s, dv_s), accumulate_dq=True)
        kd, vd = to_device(xk["k"][:, :, a:b]), to_device(xk["v"][:, :, a:b])
        dq_seg, dk_d, dv_d = va.bwd(q_d, kd, vd, o.contiguous(), lse, g_d, scale,
                                    out=(dq_d, *(t.empty((B, H, b - a, d), device="cuda") for _ in range(2))),
                                    accumulate_dq=True)
        t.cuda.synchronize()
        assert t.equal(dk_s, dk_d) and t.equal(dv_s, dv_d)
        assert_close({"dk": np64(dk_s), "dv": np64(dv_s)}, {"dk": ref["dk"][:, :, a:b], "dv": ref["dv"][:, :, a:b]},
                     names=("dk", "dv"), label=f"segment {a}:{b} d={d}")
    assert t.equal(dq_s, dq_d)
    assert_close({"o": np64(o), "lse": np64(lse), "dq": np64(dq_s)}, ref, names=("o", "lse", "dq"),
                 label=f"strided segments d={d}")


@pytest.mark.parametrize("d,H", [(72, 2), (160, 1)])
def test_paper_head_dims_at_16k_tokens(d, H):
    """N = 16,384 at the paper's other head dims: ViT-10B (d = 72, two of its
    64 heads) and the Sec. V-C model (d = 160, one of 16 heads per rank at 16
    Ulysses ranks); head (0, 0) compared in full, and the run repeated for
    bitwise determinism."""
    t = torch()
    N = 16384
    print(f"case N={N} d={d} H={H}", flush=True)
    x = workloads.make_small_inputs(1, H, N, d, seed=3100 + d)
    scale = 1.0 / np.sqrt(d)
    res = dense_run(x, scale)
    again = dense_run(x, scale)
    for n in res:
        assert t.equal(res[n], again[n]), f"{n} is not deterministic"
    ref = oracle.forward_backward(x["q"], x["k"], x["v"], x["dout"], scale, heads=[(0, 0)])
    got = {n: np64(v[0, 0]) for n, v in res.items()}
    assert_close(got, {n: a[0, 0] for n, a in ref.items()}, label=f"N={N} d={d} head (0,0)")


def _pitched_input(bits, pitch):
    """bf16 bits [1, 1, N, d] placed in rows `pitch` elements apart, NaN
    between them (a read of it would poison the outputs); returns the
    [1, 1, N, d] view."""
    t = torch()
    N, d = bits.shape[2], bits.shape[3]
    buf = t.full((N, pitch), float("nan"), dtype=t.bfloat16, device="cuda")
    buf[:, :d] = to_device(bits)[0, 0]
    return buf[:, :d][None, None]


def test_largest_input_pitch_and_outputs_past_4_gib():
    """Input rows as far apart as the library allows ((N + 256) * row * 2 bytes
    just below 2^31: the kernels address one head's rows with 32-bit offsets)
    and fp32 output rows spanning more than 2^32 bytes (64-bit offsets): every
    output bitwise equal to the dense call's, nothing written between the
    output rows, and all five outputs against the oracle element by element."""
    t = torch()
    B, H, N, d = 1, 1, 7937, 8
    pitch_in, pitch_out = 131056, 135304
    assert (N + 256) * pitch_in * 2 < 2**31 <= (N + 256) * (pitch_in + 8) * 2
    assert N * pitch_out * 4 > 2**32
    print(f"case largest pitch N={N} d={d} in={pitch_in} out={pitch_out}", flush=True)
    x = workloads.make_small_inputs(B, H, N, d, seed=1900)
    scale = 1.0 / np.sqrt(d)
    ins = [_pitched_input(x[n], pitch_in) for n in ("q", "k", "v", "dout")]
    sentinel = 12345.0
    bufs = [t.full((N, pitch_out), sentinel, dtype=t.float32, device="cuda") for _ in range(4)]  # o dq dk dv
    outs = (bufs[0][:, :d][None, None], t.empty((B, H, N), dtype=t.float32, device="cuda"),
            *(b[:, :d][None, None] for b in bufs[1:]))
    res = run(*ins, scale, outs=outs)
    dense = dense_run(x, scale)
    for n in res:
        assert t.equal(res[n], dense[n]), f"{n} differs bitwise from the dense layout"
    for name, b in zip(("o", "dq", "dk", "dv"), bufs):
        assert int(t.count_nonzero(b != sentinel)) == N * d, f"{name}: a write missed its row or left it"
    got = {n: np64(v) for n, v in res.items()}
    del ins, bufs, outs, res
    t.cuda.empty_cache()
    assert_close(got, oracle.forward_backward(x["q"], x["k"], x["v"], x["dout"], scale), label="largest pitch")


def test_longest_sequence_at_a_16_kib_pitch():
    """N = 130,815 input rows 16 KB apart, the longest sequence the 32-bit
    offsets allow at that pitch, with ragged last tiles: bitwise equal to the
    dense call; sampled query rows (O, LSE, dQ) against the oracle; dK and dV
    through identities that hold at any size (dS rows sum to zero, so the
    dK rows sum to zero; P rows sum to one, so the dV rows sum to the dO
    rows' sum)."""
    t = torch()
    B, H, N, d, pitch = 1, 1, 130815, 8, 8192
    assert (N + 256) * pitch * 2 < 2**31 <= (N + 257) * pitch * 2
    print(f"case longest sequence N={N} d={d} pitch={pitch}", flush=True)
    x = workloads.make_small_inputs(B, H, N, d, seed=1901)
    scale = 1.0 / np.sqrt(d)
    ins = [_pitched_input(x[n], pitch) for n in ("q", "k", "v", "dout")]
    res = run(*ins, scale)
    del ins
    t.cuda.empty_cache()
    dense = dense_run(x, scale)
    for n in res:
        assert t.equal(res[n], dense[n]), f"{n} differs bitwise from the dense layout"
    rng = np.random.default_rng(1901)
    idx = np.unique(np.concatenate([[0, N - 1], rng.choice(N, 62, replace=False)]))
    rows = np.stack([np.zeros_like(idx), np.zeros_like(idx), idx], axis=1)
    ref = oracle.query_rows(x["q"], x["k"], x["v"], scale, rows, dout=x["dout"])
    sel = tuple(t.from_numpy(rows[:, i]).cuda() for i in range(3))
    assert_close({n: np64(res[n][sel]) for n in ("o", "lse", "dq")}, ref, names=("o", "lse", "dq"),
                 label="longest sequence sampled query rows")
    dk, dv, g = res["dk"][0, 0].double(), res["dv"][0, 0].double(), to_device(x["dout"])[0, 0].double()
    r_dk = (dk.sum(0).norm() / dk.norm()).item()
    r_dv = ((dv.sum(0) - g.sum(0)).norm() / dv.norm()).item()
    print("longest sequence identities", {"sum_dk": r_dk, "sum_dv": r_dv}, flush=True)
    assert r_dk < 1e-2 and r_dv < 1e-2
