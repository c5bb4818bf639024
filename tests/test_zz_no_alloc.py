"""The allocation-free evaluator (redash_eval_scale_noalloc) against
redash_eval_scale, which takes a caller-provided working buffer: two calls in
a row on one GPU, the second smaller and on another base, each compared word
for word and decoded.  The second call finds the first call's contents in the
fixed buffer."""

from __future__ import annotations

import numpy as np
import pytest

torch = pytest.importorskip("torch")

from paper_2506_14489_amd import binding as B  # noqa: E402
from paper_2506_14489_amd import workloads as WL  # noqa: E402

pytestmark = pytest.mark.gpu

if not torch.cuda.is_available():  # pragma: no cover - CPU containers
    pytest.skip("needs a GPU", allow_module_level=True)


def _eval_both(w):
    x = WL.make_inputs(w)
    params = B.make_params(w.moduli, w.scale_idx, len(x), w.seed)
    sz = B.redash_plan(params)
    assert sz["work_words"] <= B.NOALLOC_WORK_WORDS  # n times the words per gadget
    print(f"noalloc: {w.name}, {len(x)} gadgets, {sz['work_words']} working words", flush=True)
    buf = B.Buffers(params, "cuda")
    B.redash_garble_scale(params, buf.offsets, buf.in_zero, buf.out_zero, buf.tables, buf.work)
    B.redash_encode(params, torch.from_numpy(x).cuda(), buf.in_zero, buf.offsets, buf.in_labels)
    B.redash_eval_scale(params, buf.in_labels, buf.tables, buf.out_labels, buf.work)
    out = torch.full_like(buf.out_labels, -1)
    B.redash_eval_scale_noalloc(params, buf.in_labels, buf.tables, out)
    B.redash_decode(params, out, buf.out_zero, buf.offsets, buf.y, buf.bad)
    torch.cuda.synchronize()
    assert torch.equal(out, buf.out_labels), f"{w.name}: labels differ from redash_eval_scale"
    assert int(buf.bad.item()) == 0
    assert np.array_equal(buf.y.cpu().numpy()[: len(x)], np.floor_divide(x, w.s))
    del buf, out
    torch.cuda.empty_cache()


def test_noalloc_matches_eval_scale_two_calls():
    # 200,704 gadgets of a ResNet-18 layer-1 conv on the 12-prime base (a full
    # round on 2 waves per 64 gadgets and the rest on 12, one launch), then
    # the 65,536 of the 10-prime conv map scaled by 23 * 29 (a smaller call:
    # 4 waves per 64 gadgets)
    _eval_both(WL.by_name("resnet18.l1.1.a"))
    _eval_both(WL.CONV)


def test_noalloc_under_graph_capture():
    """The callers it is for: captured in a graph, then three replays with
    eager calls and synchronizations between them; every replay equals
    redash_eval_scale on a caller-provided working buffer."""
    w = WL.by_name("resnet18.l2.0.b")
    x = WL.make_inputs(w)
    params = B.make_params(w.moduli, w.scale_idx, len(x), w.seed)
    print(f"noalloc under capture: {w.name}, {len(x)} gadgets", flush=True)
    buf = B.Buffers(params, "cuda")
    B.redash_garble_scale(params, buf.offsets, buf.in_zero, buf.out_zero, buf.tables, buf.work)
    B.redash_encode(params, torch.from_numpy(x).cuda(), buf.in_zero, buf.offsets, buf.in_labels)
    B.redash_eval_scale(params, buf.in_labels, buf.tables, buf.out_labels, buf.work)
    torch.cuda.synchronize()
    ref = buf.out_labels.clone()
    out_g = torch.full_like(ref, -1)
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g, capture_error_mode="thread_local"):
        B.redash_eval_scale_noalloc(params, buf.in_labels, buf.tables, out_g)
    for _ in range(3):
        out_g.fill_(-1)
        torch.cuda.synchronize()
        g.replay()
        B.redash_eval_scale(params, buf.in_labels, buf.tables, buf.out_labels, buf.work)
        torch.cuda.synchronize()
        assert torch.equal(out_g, ref)
        assert torch.equal(buf.out_labels, ref)
    B.redash_decode(params, out_g, buf.out_zero, buf.offsets, buf.y, buf.bad)
    torch.cuda.synchronize()
    assert int(buf.bad.item()) == 0
    assert np.array_equal(buf.y.cpu().numpy()[: len(x)], np.floor_divide(x, w.s))
    del g, buf, out_g, ref
    torch.cuda.empty_cache()
