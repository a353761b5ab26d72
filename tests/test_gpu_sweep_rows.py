"""Seeded random sweeps of the rows beside the attention: the channel
aggregation (random M, H, C, d) against its oracle element by element, the
Ulysses layout copies (random B, Nl, H, P, row size, dtype) bit-exactly
against the oracle's index maps, and key segments at random cuts merged and
compared with the oracle's attention over all keys."""
import numpy as np
import pytest

import oracle
from oracle import aggregation as agg
from oracle import ulysses as uref
import workloads
from gpu_util import TOL_GRAD_REL, TOL_LSE_MAX, TOL_O_MAX, TOL_O_REL, assert_close, rel_l2, to_device, torch

pytestmark = pytest.mark.gpu


def np64(t):
    return t.detach().double().cpu().numpy()


@pytest.mark.parametrize("seed", [1, 2])
def test_random_aggregation_calls_match_the_oracle(seed):
    import paper_2405_15780_amd as va

    rng = np.random.default_rng(seed)
    for case in range(12):
        M, H, C = int(rng.integers(1, 300)), int(rng.integers(1, 9)), int(rng.integers(1, 260))
        d = int(rng.choice([64, 128]))
        print(f"seed {seed} case {case}: M={M} H={H} C={C} d={d}", flush=True)
        x = workloads.make_aggregation_inputs(M, H, C, d, seed=1000 * seed + case)
        dev = {n: to_device(a) for n, a in x.items()}
        scale = 1.0 / np.sqrt(d)
        o, lse = va.agg_fwd(dev["q"], dev["k"], dev["v"], scale)
        dq, dk, dv = va.agg_bwd(dev["q"], dev["k"], dev["v"], o, lse, dev["dout"], scale)
        torch().cuda.synchronize()
        ref = agg.backward(x["q"], x["k"], x["v"], x["dout"], scale)
        g = {"o": np64(o), "lse": np64(lse), "dq": np64(dq), "dk": np64(dk), "dv": np64(dv)}
        assert float(np.abs(g["o"] - ref["o"]).max()) <= TOL_O_MAX and rel_l2(g["o"], ref["o"]) <= TOL_O_REL
        assert float(np.abs(g["lse"] - ref["lse"]).max()) <= TOL_LSE_MAX
        for n in ("dq", "dk", "dv"):
            if np.linalg.norm(ref[n]) == 0.0:  # C = 1: p = 1 and ds = 0 exactly
                assert float(np.abs(g[n]).max()) <= 1e-5, n
            else:
                assert rel_l2(g[n], ref[n]) <= TOL_GRAD_REL, (n, rel_l2(g[n], ref[n]))


def _host(shape, dt, rng):
    if dt == "bf16":
        return rng.integers(0, 2 ** 16, size=shape, dtype=np.uint16)
    return rng.standard_normal(shape).astype(np.float32)


def _dev(a):
    t = torch()
    if a.dtype == np.uint16:
        return t.from_numpy(a.view(np.int16)).view(t.bfloat16).cuda()
    return t.from_numpy(a).cuda()


def _np(x):
    t = torch()
    a = x.cpu()
    return a.view(t.int16).numpy().view(np.uint16) if a.dtype == t.bfloat16 else a.numpy()


@pytest.mark.parametrize("seed", [1, 2])
def test_random_ulysses_copies_match_the_index_maps(seed):
    import paper_2405_15780_amd as va

    rng = np.random.default_rng(seed)
    for case in range(16):
        P = int(rng.integers(1, 9))
        B, Nl, H = int(rng.integers(1, 4)), int(rng.integers(1, 70)), P * int(rng.integers(1, 5))
        dt = str(rng.choice(["bf16", "f32"]))
        e = 8 * int(rng.integers(1, 21)) if dt == "bf16" else 4 * int(rng.integers(1, 41))
        print(f"seed {seed} case {case}: B={B} Nl={Nl} H={H} P={P} row={e} {dt}", flush=True)
        x = _host((B, Nl, H, e), dt, rng)
        send = va.ulysses_pack(_dev(x), P)
        assert np.array_equal(_np(send), uref.pack(x, P))
        recv = _host((P, B, H // P, Nl, e), dt, rng)
        y = va.ulysses_unpack(_dev(recv))
        assert np.array_equal(_np(y), uref.unpack(recv))
        back = va.ulysses_pack_out(y, P)
        assert np.array_equal(_np(back), uref.pack_out(uref.unpack(recv), P))
        xb = va.ulysses_unpack_out(send)
        assert np.array_equal(_np(xb), uref.unpack_out(uref.pack(x, P)))


@pytest.mark.parametrize("seed", [1, 2])
def test_random_key_segments_merge_to_full_attention(seed):
    import paper_2405_15780_amd as va

    t = torch()
    rng = np.random.default_rng(seed)
    for case in range(8):
        B, H = int(rng.integers(1, 3)), int(rng.integers(1, 4))
        Nq, N = int(rng.integers(1, 400)), int(rng.integers(2, 900))
        d = int(rng.choice(np.arange(8, 161, 8)))
        n_cuts = int(rng.integers(1, min(7, N)))
        cuts = sorted(set(int(c) for c in rng.integers(1, N, size=n_cuts)))
        edges = [0] + cuts + [N]
        print(f"seed {seed} case {case}: B={B} H={H} Nq={Nq} N={N} d={d} segments={len(edges) - 1}", flush=True)
        xq = workloads.make_small_inputs(B, H, Nq, d, seed=5000 * seed + 2 * case, with_dout=False)
        xk = workloads.make_small_inputs(B, H, N, d, seed=5000 * seed + 2 * case + 1, with_dout=False)
        scale = 1.0 / np.sqrt(d)
        q = to_device(xq["q"])
        parts = [va.fwd(q, to_device(np.ascontiguousarray(xk["k"][:, :, a:b])),
                        to_device(np.ascontiguousarray(xk["v"][:, :, a:b])), scale)
                 for a, b in zip(edges[:-1], edges[1:])]
        o, lse = va.merge(t.stack([p[0] for p in parts]).contiguous(), t.stack([p[1] for p in parts]).contiguous())
        t.cuda.synchronize()
        ref_o, ref_lse = oracle.forward(xq["q"], xk["k"], xk["v"], scale)
        assert_close({"o": np64(o), "lse": np64(lse)}, {"o": ref_o, "lse": ref_lse}, names=("o", "lse"),
                     label=f"seed {seed} case {case}")
