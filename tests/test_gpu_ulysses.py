"""GPU checks of the Ulysses layout kernels: each copy against the oracle's
index maps (bit-exact), and one simulated Ulysses attention pass over P ranks
(sequence-sharded Q, K, V -> pack -> all-to-all -> unpack -> attention per
rank -> pack_out -> all-to-all -> unpack_out) against the oracle's attention
of the unsharded tensors."""
import numpy as np
import pytest

import oracle
from oracle import ulysses as ref
import workloads
from gpu_util import assert_close, torch

pytestmark = pytest.mark.gpu

SHAPES = [  # B, Nl, H, P, row elements, dtype
    (1, 5, 4, 2, 64, "bf16"), (2, 33, 8, 4, 128, "bf16"), (1, 1, 3, 3, 72, "bf16"), (2, 7, 6, 1, 8, "bf16"),
    (1, 129, 4, 4, 128, "f32"), (3, 2, 2, 2, 4, "f32"),
]


def _host(B, Nl, H, P, e, dt, seed):
    rng = np.random.default_rng(seed)
    if dt == "bf16":
        return rng.integers(0, 2 ** 16, size=(B, Nl, H, e), dtype=np.uint16)
    return rng.standard_normal((B, Nl, H, e)).astype(np.float32)


def _dev(a):
    t = torch()
    if a.dtype == np.uint16:
        return t.from_numpy(a.view(np.int16)).view(t.bfloat16).cuda()
    return t.from_numpy(a).cuda()


def _np(t):
    t_ = torch()
    a = t.cpu()
    return a.view(t_.int16).numpy().view(np.uint16) if a.dtype == t_.bfloat16 else a.numpy()


@pytest.mark.parametrize("B,Nl,H,P,e,dt", SHAPES)
def test_layout_copies_match_the_oracle(B, Nl, H, P, e, dt):
    import paper_2405_15780_amd as va

    print(f"case B={B} Nl={Nl} H={H} P={P} row={e} {dt}", flush=True)
    x = _host(B, Nl, H, P, e, dt, seed=B * 1000 + Nl * 10 + H + P)
    send = va.ulysses_pack(_dev(x), P)
    assert np.array_equal(_np(send), ref.pack(x, P))
    y = va.ulysses_unpack(send)
    assert np.array_equal(_np(y), ref.unpack(_np(send)))
    back = va.ulysses_pack_out(y, P)
    assert np.array_equal(_np(back), ref.pack_out(_np(y), P))
    xx = va.ulysses_unpack_out(back)
    assert np.array_equal(_np(xx), ref.unpack_out(_np(back)))


@pytest.mark.parametrize("P,H,Nl,d", [(2, 4, 300, 64), (4, 4, 129, 128)])
def test_simulated_ulysses_attention_pass(P, H, Nl, d):
    import paper_2405_15780_amd as va

    t = torch()
    print(f"case P={P} H={H} Nl={Nl} d={d}", flush=True)
    B, N = 1, P * Nl
    # global inputs [B, H, N, d] as the oracle sees them; rank r holds tokens r*Nl.. in [B, Nl, H, d]
    x = workloads.make_small_inputs(B, H, N, d, seed=900 + P + d, with_dout=False)
    shards = {n: [np.ascontiguousarray(x[n][:, :, r * Nl:(r + 1) * Nl].transpose(0, 2, 1, 3)) for r in range(P)]
              for n in ("q", "k", "v")}
    heads = {}
    for n in ("q", "k", "v"):
        sends = [va.ulysses_pack(_dev(s), P) for s in shards[n]]
        recvs = [t.stack([sends[r][p] for r in range(P)]).contiguous() for p in range(P)]  # the all-to-all
        heads[n] = [va.ulysses_unpack(rv) for rv in recvs]  # rank p: [B, H/P, N, d]
    scale = 1.0 / np.sqrt(d)
    outs = [va.fwd(heads["q"][p], heads["k"][p], heads["v"][p], scale)[0] for p in range(P)]  # fp32 [B, H/P, N, d]
    sends = [va.ulysses_pack_out(o, P) for o in outs]
    recvs = [t.stack([sends[p][r] for p in range(P)]).contiguous() for r in range(P)]
    o_shards = [va.ulysses_unpack_out(rv) for rv in recvs]  # rank r: [B, Nl, H, d]
    t.cuda.synchronize()
    got = np.concatenate([s.double().cpu().numpy() for s in o_shards], axis=1).transpose(0, 2, 1, 3)
    ref_o, _ = oracle.forward(x["q"], x["k"], x["v"], scale)
    assert_close({"o": got}, {"o": ref_o}, names=("o",), label=f"ulysses P={P} H={H} N={N} d={d}")
