"""GPU test of peek_queue_signals_noalloc (the queue signals with the
library's static scratch): called through the C ABI, its outputs must equal
those of peek_queue_signals with a caller's workspace, element by element,
on two calls in a row, the second with a smaller queue, anchored on the walk
and from scratch."""
import numpy as np
import pytest

import oracle as O
import peek_workloads as W

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")


def _signals_pair(P, hp, n, anchored):
    """Outputs of both entry points on the first n requests of the queue."""
    i32 = torch.int32
    dev = hp.device
    off = hp.d_offsets[:n + 1]
    last = hp.d_last[:n] if n else hp.d_last[:1]
    m = hp.d_m[:n] if (anchored and n) else (hp.d_m[:1] if anchored else None)
    ws = torch.empty(max(P.peek_queue_signals_workspace(n, hp.num_nodes), 256), dtype=torch.uint8, device=dev)
    out = {}
    for kind in ("workspace", "static"):
        cid = torch.full((max(n, 1),), -7, dtype=i32, device=dev)
        csz = torch.full((max(n, 1),), -7, dtype=i32, device=dev)
        dem = torch.full((hp.num_nodes,), -7, dtype=i32, device=dev)
        if kind == "workspace":
            P.peek_queue_signals(hp.cache, hp.d_tokens, off, last, m, hp.threshold, cid, csz, dem, ws)
        else:
            P.peek_queue_signals_noalloc(hp.cache, hp.d_tokens, off, last, m, hp.threshold, cid, csz, dem)
        torch.cuda.synchronize()
        out[kind] = (cid[:n].cpu().numpy(), csz[:n].cpu().numpy(), dem.cpu().numpy())
    return out


@pytest.mark.parametrize("name", ["rag", "agentic"])
def test_noalloc_signals_match_the_workspace_entry_point(name):
    import paper_2607_02525_amd as P
    from paper_2607_02525_amd.runner import HotPath
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    w = W.make(name, 42)
    hp = HotPath.from_sequences(*w.cache_sequences)
    hp.load_queue(w.tokens, w.offsets, w.block_size, w.threshold)
    hp.lpm()
    torch.cuda.synchronize()
    s = O.run(w)
    # two calls in a row, the second with a smaller queue (the static scratch
    # then holds the first call's contents)
    for n in (w.n, w.n // 3):
        for anchored in (True, False):
            print(f"[gpu] noalloc {name} n={n} anchored={anchored}", flush=True)
            out = _signals_pair(P, hp, n, anchored)
            for a, b, what in zip(out["workspace"], out["static"], ("cluster_id", "cluster_size", "demand")):
                assert np.array_equal(a, b), f"{what} differs (n={n}, anchored={anchored})"
            if n == w.n:
                assert np.array_equal(out["static"][0], s.clusters.cluster_id)
                assert np.array_equal(out["static"][1], s.clusters.cluster_size)
                assert np.array_equal(out["static"][2], s.demand)
