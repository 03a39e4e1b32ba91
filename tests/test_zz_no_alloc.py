"""The allocation-free measurement call (ckv_measure_page_effects_noalloc)
against the regular call on the same inputs, through the C ABI: two calls in
a row, the second on a smaller problem, each compared with
ckv_measure_page_effects (R and R_head within 2e-3 relative, o, lse and the
token mass within float32 summation-order differences)."""
import numpy as np
import pytest
import torch

from synth import WORKLOADS, make_layer
from tests.gpu_util import LayerOnDevice, assert_scores_close

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ckv():
    import paper_2608_07855_amd as P
    ctx = P.Context(0)
    yield P, ctx
    ctx.close()


def _random_problem(S, Hq, Hkv, W, d, n_pages, seed):
    g = torch.Generator(device="cuda").manual_seed(seed)
    k = torch.randn(Hkv, S, d, device="cuda", generator=g).to(torch.bfloat16)
    v = torch.randn(Hkv, S, d, device="cuda", generator=g).to(torch.bfloat16)
    q = torch.randn(Hq, W, d, device="cuda", generator=g).to(torch.bfloat16)
    pos = torch.arange(S, dtype=torch.int32, device="cuda")
    qpos = torch.arange(S - W, S, dtype=torch.int32, device="cuda")
    starts = np.arange(n_pages, dtype=np.int32) * 48 + 100
    lens = np.full(n_pages, 32, np.int32)
    return k, v, q, pos, qpos, starts, lens


def _compare(P, ctx, kv, win, pages, what):
    want = ("R", "R_head", "o", "lse", "token_mass")
    ref = P.ckv_measure_page_effects(ctx, kv, win, pages, want=want)
    got = P.ckv_measure_page_effects(ctx, kv, win, pages, want=want, noalloc=True)
    torch.cuda.synchronize()
    print(f"[noalloc] {what}: {pages.n} pages", flush=True)
    assert_scores_close(got["R"].cpu().numpy(), ref["R"].cpu().numpy(), f"{what} R")
    assert_scores_close(got["R_head"].cpu().numpy(), ref["R_head"].cpu().numpy(), f"{what} R_head")
    np.testing.assert_allclose(got["o"].cpu().numpy(), ref["o"].cpu().numpy(), rtol=1e-4, atol=1e-5)
    np.testing.assert_allclose(got["lse"].cpu().numpy(), ref["lse"].cpu().numpy(), rtol=1e-5, atol=1e-5)
    np.testing.assert_allclose(got["token_mass"].cpu().numpy(), ref["token_mass"].cpu().numpy(),
                               rtol=1e-4, atol=1e-7)


def test_noalloc_matches_regular_call(ckv):
    P, ctx = ckv
    # 1024 window rows per KV head: the regular call's split partials do not
    # fit the 64 MiB scratch, so the allocation-free call takes fewer splits
    k, v, q, pos, qpos, starts, lens = _random_problem(40000, 64, 8, 128, 128, 700, seed=7)
    kv = P.kv_view(k, v, pos)
    win = P.window_view(q, qpos)
    _compare(P, ctx, kv, win, P.Pages(starts, lens), "40000 tokens, 8192 rows")
    # then a smaller problem on the same scratch
    L = make_layer(WORKLOADS["tiny"], seed=4)
    dl = LayerOnDevice(L)
    kv2 = P.kv_view(dl.k, dl.v, dl.pos)
    win2 = P.window_view(dl.q_post, dl.qpos_post)
    _compare(P, ctx, kv2, win2, P.Pages(L.layout.page_start, L.layout.page_len), "tiny")


def test_noalloc_rejects_oversized_shape(ckv):
    """A shape whose working memory exceeds the scratch even with one split
    fails on the host with CKV_ERR_UNSUPPORTED and enqueues nothing."""
    P, ctx = ckv
    S, Hq, Hkv, W, d = 4096, 128, 8, 1024, 128    # 131072 window rows
    k = torch.zeros(Hkv, S, d, dtype=torch.bfloat16, device="cuda")
    q = torch.zeros(Hq, W, d, dtype=torch.bfloat16, device="cuda")
    pos = torch.arange(S, dtype=torch.int32, device="cuda")
    qpos = torch.arange(S, S + W, dtype=torch.int32, device="cuda")
    kv = P.kv_view(k, k, pos)
    win = P.window_view(q, qpos)
    with pytest.raises(P.CKVError) as e:
        P.ckv_measure_page_effects(ctx, kv, win, P.Pages([0], [16]), noalloc=True)
    assert e.value.code == -4
