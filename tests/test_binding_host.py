"""Host-side argument checks of the Python binding: tensors that are not on
a GPU are rejected with TypeError before any library call, and without the
built library every call raises (there is no fallback)."""
import pytest

torch = pytest.importorskip("torch")

import paper_2405_15780_amd as va


def bf16(*shape):
    return torch.zeros(shape, dtype=torch.bfloat16)


def test_attention_rejects_host_tensors():
    q = bf16(1, 2, 8, 64)
    with pytest.raises(TypeError):
        va.fwd(q, q, q)
    o, lse = torch.zeros(1, 2, 8, 64), torch.zeros(1, 2, 8)
    with pytest.raises(TypeError):
        va.bwd(q, q, q, o, lse, q)


def test_stage_entry_points_reject_host_tensors():
    q = bf16(1, 2, 8, 64)
    f = torch.zeros(1, 2, 8, 64)
    lse = torch.zeros(1, 2, 8)
    ws = torch.zeros(1 << 16)
    with pytest.raises(TypeError):
        va.bwd_rowdot(f, q, lse, ws)
    with pytest.raises(TypeError):
        va.bwd_dkdv(q, q, q, q, lse, f, f, ws)
    with pytest.raises(TypeError):
        va.bwd_dq(q, q, q, q, lse, f, ws)
    with pytest.raises(TypeError):
        va.bwd_dkdv_ds(q, q, q, q, lse, f, f, ws)
    with pytest.raises(TypeError):
        va.bwd_dq_from_ds(q, f, ws)


def test_other_rows_reject_host_tensors():
    with pytest.raises(TypeError):
        va.merge(torch.zeros(2, 1, 2, 8, 64), torch.zeros(2, 1, 2, 8))
    with pytest.raises(TypeError):
        va.agg_fwd(bf16(2, 64), bf16(3, 2, 5, 64), bf16(3, 2, 5, 64))
    with pytest.raises(TypeError):
        va.ulysses_pack(bf16(1, 8, 4, 64), 2)


def test_missing_library_raises_instead_of_falling_back(monkeypatch):
    # there is no CPU or PyTorch path: without the built library every call
    # that needs it raises
    from paper_2405_15780_amd import binding

    monkeypatch.setattr(binding, "_lib", None)
    monkeypatch.setattr(binding, "LIB_PATH", "/nonexistent/libvitattn.so")
    with pytest.raises(ImportError, match="is missing"):
        binding.library()
    with pytest.raises(ImportError, match="is missing"):
        binding.workspace_bytes(1, 1, 8, 64)
    with pytest.raises(ImportError, match="is missing"):
        binding.version()
