"""hb_predict_scratch, the entry point that allocates nothing, against
hb_predict_ws with a caller workspace of the same size: two calls in a row on
one GPU, the second with fewer rows, both taking the tree split whose partial
sums live in the scratch. Leaf ids must be identical and scores within
1e-5 (1 + |reference|); the kernels and the split are the same, so they are
expected bit for bit."""
import numpy as np
import pytest

import paper_2010_04804_amd as hb
from paper_2010_04804_amd import synth

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def say(*a):
    print("[case]", *a, flush=True)


@pytest.fixture(scope="module", autouse=True)
def need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")


def _pair(h, X, strategy, nbytes):
    n = X.shape[0]
    info = h.info()
    dev = X.device
    out = []
    for scratch in (False, True):
        scores = torch.full((n, info["n_outputs"]), float("nan"), dtype=torch.float32, device=dev)
        ids = torch.full((n, info["n_trees"]), -7, dtype=torch.int32, device=dev)
        stream = torch.cuda.current_stream(dev).cuda_stream
        if scratch:
            hb.predict_scratch_ptr(h, X.data_ptr(), n, scores.data_ptr(), ids.data_ptr(), strategy, stream, nbytes)
        else:
            ws = torch.empty(max(nbytes, 8), dtype=torch.uint8, device=dev)
            hb.predict_ptr(h, X.data_ptr(), n, scores.data_ptr(), ids.data_ptr(), strategy, stream,
                           ws.data_ptr(), nbytes)
        torch.cuda.synchronize()
        out.append((scores.cpu().numpy(), ids.cpu().numpy()))
    return out


@pytest.mark.parametrize("cfg,strategy,sizes", [(2, "ptt", (40_000, 3_000)), (5, "tt", (20_000, 1_500)),
                                                (4, "ptt", (8_000, 2_049))])
def test_scratch_matches_workspace(cfg, strategy, sizes):
    model = synth.make_model(cfg)
    h = hb.compile(model, device=0)
    for n in sizes:  # two calls in a row, the second smaller
        nbytes = min(hb.workspace_bytes(h, n, strategy), hb.SCRATCH_BYTES)
        plan = h.plan(n, strategy, nbytes)
        say("scratch", cfg, strategy, n, nbytes, [p["kernel"] for p in plan])
        assert nbytes > 0 and any("split_finish" in p["kernel"] for p in plan), "the call must use the scratch"
        X = torch.from_numpy(synth.make_rows(cfg, n)).cuda()
        (s_ws, i_ws), (s_sc, i_sc) = _pair(h, X, strategy, nbytes)
        assert np.array_equal(i_sc, i_ws), f"cfg{cfg}/{strategy}/{n}: leaf ids differ"
        err = np.abs(s_sc.astype(np.float64) - s_ws)
        assert np.all(err <= 1e-5 * (1 + np.abs(s_ws))), f"cfg{cfg}/{strategy}/{n}: max err {err.max()}"
        assert np.array_equal(s_sc, s_ws)
    h.close()


def test_scratch_rejects_sizes_beyond_the_maximum():
    h = hb.compile(synth.make_model(1), device=0)
    X = torch.zeros((10, 8), dtype=torch.float32, device="cuda")
    s = torch.empty((10, 1), dtype=torch.float32, device="cuda")
    say("scratch oversize")
    with pytest.raises(hb.HBError) as e:
        hb.predict_scratch_ptr(h, X.data_ptr(), 10, s.data_ptr(), None, "ptt", None, hb.SCRATCH_BYTES + 1)
    assert e.value.code == -1 and "HB_SCRATCH_BYTES" in str(e.value)
    h.close()
