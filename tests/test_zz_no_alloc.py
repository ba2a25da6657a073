"""sv_spec_accept_noalloc against sv_spec_accept: the same kernels with the library's fixed
device scratch in place of the caller's workspace, so every output must match bit for bit.
Two calls in a row on the scratch, the second on a smaller input, in both input kinds."""
import numpy as np
import pytest

from gpu_util import say

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    from paper_2607_25852_amd import binding
    binding.load()
    return torch


def _round(torch, seed, R, b, V, kind):
    """Seeded device inputs of one acceptance call: ragged packing, logits (bf16) or
    probability rows (fp32), drafted tokens, uniforms on the 2^-24 grid."""
    g = torch.Generator(device="cuda").manual_seed(seed)
    rng = np.random.default_rng(seed)
    D = b - 1
    k = rng.integers(1, b + 1, size=R)
    qo = np.concatenate([[0], np.cumsum(k)]).astype(np.int32)
    K = int(qo[-1])
    if kind == "logits":
        tgt = torch.randn((K, V), generator=g, device="cuda") * 3.0
        dr = torch.randn((R, max(D, 1), V), generator=g, device="cuda") * 3.0
        tgt, dr = tgt.to(torch.bfloat16), dr[:, :D].contiguous().to(torch.bfloat16)
    else:
        tgt = torch.rand((K, V), generator=g, device="cuda") ** 4
        dr = torch.rand((R, max(D, 1), V), generator=g, device="cuda")[:, :D].contiguous() ** 4
        tgt = tgt / tgt.sum(-1, keepdim=True)
        dr = (dr / dr.sum(-1, keepdim=True)).contiguous()
    toks = torch.from_numpy(rng.integers(0, V, size=(R, D)).astype(np.int32)).cuda()
    ua = torch.from_numpy((rng.integers(0, 1 << 24, size=(R, D)) * 2.0 ** -24).astype(np.float32)).cuda()
    us = torch.from_numpy((rng.integers(0, 1 << 24, size=R) * 2.0 ** -24).astype(np.float32)).cuda()
    return dict(target=tgt, draft=dr, toks=toks, qo=torch.from_numpy(qo).cuda(), ua=ua, us=us, R=R, b=b, V=V,
                kind=kind)


def _outputs(torch, r):
    return (torch.full((r["R"],), -9, dtype=torch.int32, device="cuda"),
            torch.full((r["R"], r["b"]), -9, dtype=torch.int32, device="cuda"),
            torch.full((r["R"],), -9, dtype=torch.int32, device="cuda"))


def _desc(r):
    from paper_2607_25852_amd import binding as B
    kind = B.SV_LOGITS if r["kind"] == "logits" else B.SV_PROBS
    dtype = B.SV_BF16 if r["kind"] == "logits" else B.SV_F32
    return B.accept_desc(r["R"], r["b"], r["V"], kind, dtype, 1.0)


def _with_workspace(torch, r):
    from paper_2607_25852_amd import binding as B
    d = _desc(r)
    ws = torch.empty(B.accept_workspace_size(d), dtype=torch.uint8, device="cuda")
    acc, out, fl = _outputs(torch, r)
    B.spec_accept(d, r["target"], r["draft"], r["toks"], r["qo"], r["ua"], r["us"], acc, out, fl, ws)
    torch.cuda.synchronize()
    return acc.cpu().numpy(), out.cpu().numpy(), fl.cpu().numpy()


def _no_alloc(torch, r):
    from paper_2607_25852_amd import binding as B
    acc, out, fl = _outputs(torch, r)
    B.spec_accept_noalloc(_desc(r), r["target"], r["draft"], r["toks"], r["qo"], r["ua"], r["us"], acc, out, fl)
    torch.cuda.synchronize()
    return acc.cpu().numpy(), out.cpu().numpy(), fl.cpu().numpy()


@pytest.mark.parametrize("kind", ["logits", "probs"])
def test_noalloc_equals_workspace_call_twice(dev, kind):
    from paper_2607_25852_amd import binding as B
    big = (64, 16, 131072) if kind == "logits" else (64, 16, 32768)
    shapes = [big, (9, 5, 40001)]  # the second call is smaller than the first
    for n, (R, b, V) in enumerate(shapes):
        r = _round(dev, 1000 + n + (7 if kind == "probs" else 0), R, b, V, kind)
        assert B.accept_workspace_size(_desc(r)) <= 16 << 20
        say("noalloc", kind, "call", n, "R", R, "b", b, "V", V)
        ref = _with_workspace(dev, r)
        got = _no_alloc(dev, r)
        for x, y in zip(got, ref):
            np.testing.assert_array_equal(x, y)
        assert np.all(ref[0] >= 0) and np.all(ref[0] <= np.diff(r["qo"].cpu().numpy()) - 1)


def test_noalloc_rejects_oversized_shapes(dev):
    from paper_2607_25852_amd import binding as B
    d = B.accept_desc(4096, 16, 131072, B.SV_LOGITS, B.SV_BF16, 1.0)  # needs far more than 16 MiB
    with pytest.raises(B.SpecVerifyError) as e:
        B.spec_accept_noalloc(d, None, None, None, None, None, None, None, None)
    assert e.value.status == B.SV_ERR_UNSUPPORTED and "16777216" in str(e.value)
