"""A step (peek_lpm_batch + peek_queue_signals) captured into a HIP graph
and replayed: the calls enqueue kernels only (no memset, copy or host wait
inside), so the graph replays the whole step. Every replay, with eager work
on the same buffers in between, must match the eagerly computed outputs."""
import numpy as np
import pytest

import peek_workloads as W

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("name", ["rag", "caterpillar"])
def test_captured_step_replays_match_eager(name):
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2607_02525_amd.runner import HotPath
    w = W.make(name, 42)
    print(f"[gpu] graph capture {name} n={w.n}", flush=True)
    hp = HotPath.from_description(*w.cache_tree) if w.cache_tree is not None else \
        HotPath.from_sequences(*w.cache_sequences)
    hp.load_queue(w.tokens, w.offsets, w.block_size, w.threshold)
    hp.step()
    ref = {k: v.copy() for k, v in hp.results().items() if isinstance(v, np.ndarray)}
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        hp.step()   # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        hp.step()
    torch.cuda.synchronize()
    for rep in range(4):
        # eager work on the output buffers between replays
        hp.d_cid.fill_(-7)
        hp.d_csz.fill_(-7)
        hp.d_demand.fill_(-7)
        hp.d_h.fill_(-7)
        torch.cuda.synchronize()
        g.replay()
        torch.cuda.synchronize()
        got = hp.results()
        for k in ref:
            assert np.array_equal(got[k], ref[k]), f"replay {rep}: {k}"
        hp.step()   # and an eager step in between, same result
        got = hp.results()
        for k in ref:
            assert np.array_equal(got[k], ref[k]), f"eager after replay {rep}: {k}"
