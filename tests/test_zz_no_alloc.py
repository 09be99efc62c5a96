"""uattn_decode_noalloc (the decode entry point that allocates nothing and
uses the library's static scratch array) against uattn_decode with a caller
workspace: the same bits, outputs and lse, on two calls in a row, the second
with a smaller batch and shorter contexts, and again after a uattn_decode
call has used its own workspace in between.  Also checks that the call can
be captured into a HIP graph and replayed with new inputs."""
import numpy as np
import pytest

from paper_2609_35140_amd import inputs

pytestmark = pytest.mark.gpu

gu = pytest.importorskip("gpu_util")


@pytest.fixture(scope="module")
def ua():
    import torch
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2609_35140_amd import uattn
    uattn.lib()
    return uattn


def _both(ua, pk, entries, label):
    import torch
    q, table, seqlens, maxs, _ = pk.decode_rows(entries)
    ref, ref_lse = ua.decode(q, pk.kp, pk.vp, table, seqlens, maxs, return_lse=True)
    # caller-allocated outputs filled with garbage: everything must be written
    out = torch.full_like(q, float("nan"))
    lse = torch.full((q.shape[0], q.shape[1]), float("nan"), dtype=torch.float32, device="cuda")
    ua.decode_noalloc(q, pk.kp, pk.vp, table, seqlens, maxs, out=out, lse=lse)
    torch.cuda.synchronize()
    same = torch.equal(out.view(torch.int16), ref.view(torch.int16))
    lse_same = torch.equal(lse.view(torch.int32), ref_lse.view(torch.int32))
    print(f"{label}: batch {len(entries)}, max ctx {maxs}: outputs bitwise {same}, lse bitwise {lse_same}", flush=True)
    assert same and lse_same, label


def test_noalloc_equals_decode_two_calls(ua):
    # Qwen-style heads (32 q / 8 kv, d 128, page 64), 8 sequences up to 4096 keys
    w = inputs.custom(32, 8, 128, [4096, 3000, 4096, 2049, 1500, 4000, 257, 3333], sigma=0.5, page_size=64)
    pk = gu.Pack(w, seed=7)
    g = inputs.rng(61, 0)
    big = [(s, int(L) - 1 - int(g.integers(0, 40))) for s, L in enumerate(w.seq_lens)]
    _both(ua, pk, big, "first call")
    # second call: fewer entries, shorter contexts (fewer chunks, smaller counter region)
    small = [(1, 700), (6, 255), (3, 1025)]
    _both(ua, pk, small, "second call (smaller)")
    # a decode with its own workspace in between, then the no-alloc path again
    _both(ua, pk, big[::-1], "third call (reversed batch)")


def test_noalloc_graph_replay(ua):
    import torch
    w = inputs.custom(16, 2, 128, [1800, 900, 2500], sigma=1.0, page_size=64)
    pk = gu.Pack(w, seed=11)
    entries = [(0, 1799), (1, 899), (2, 2499)]
    q, table, seqlens, maxs, _ = pk.decode_rows(entries)
    out = torch.empty_like(q)
    lse = torch.empty((q.shape[0], q.shape[1]), dtype=torch.float32, device="cuda")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    ua.decode_noalloc(q, pk.kp, pk.vp, table, seqlens, maxs, out=out, lse=lse, stream=s)  # first use on the device
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=s):
        ua.decode_noalloc(q, pk.kp, pk.vp, table, seqlens, maxs, out=out, lse=lse, stream=s)
    torch.cuda.synchronize()
    for rep, ent in enumerate([entries, [(0, 1000), (1, 300), (2, 2000)], [(0, 1799), (1, 0), (2, 1024)]]):
        q2, _, sl2, _, _ = pk.decode_rows(ent)
        q.copy_(q2)
        seqlens.copy_(sl2)
        out.fill_(float("nan"))
        graph.replay()
        torch.cuda.synchronize()
        ref, ref_lse = ua.decode(q, pk.kp, pk.vp, table, seqlens, maxs, return_lse=True)
        torch.cuda.synchronize()
        assert torch.equal(out.view(torch.int16), ref.view(torch.int16)), f"replay {rep}"
        assert torch.equal(lse.view(torch.int32), ref_lse.view(torch.int32)), f"replay {rep}"
    print("graph replay: 3 replays with new queries and lengths equal eager uattn_decode", flush=True)
