"""kb_screen_noalloc and kb_screen captured in a HIP graph (GPU)."""
import sys

import pytest
import torch

import paper_2608_02611_amd as kb
from tests.helpers import assert_records_match, ensure_built, oracle_records

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    ensure_built()
    return torch.device("cuda:0")


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def test_noalloc_in_a_captured_graph(dev):
    """The call for callers that cannot allocate, recorded into a graph once
    and replayed: every replay (with eager work and synchronizations between
    them, and the records cleared before each) gives the eager call's
    records, which equal the oracle's."""
    g = torch.Generator(device=dev).manual_seed(11)
    n, K = (1 << 18) + 77, 24
    ref = torch.randn(n, generator=g, device=dev).to(torch.float16)
    cands = [(ref.float() * (1 + 3e-4 * torch.randn(n, generator=g, device=dev))).to(torch.float16)
             for _ in range(K)]
    for k in range(0, K, 5):
        cands[k][(k * 7919) % n] += 2.0
    d_stats = kb.alloc_stats(K, dev)
    # eager call first: the scratch address and the occupancy are looked up once
    say("graph: eager")
    kb.kb_screen_noalloc(ref, cands, 1e-3, 1e-3, d_stats=d_stats)
    want, _ = kb.kb_screen_stats(d_stats, K)
    assert_records_match(want, oracle_records(ref, cands, 1e-3, 1e-3), "eager")
    say("graph: capture")
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        kb.kb_screen_noalloc(ref, cands, 1e-3, 1e-3, d_stats=d_stats)
    torch.cuda.synchronize()
    for i in range(4):
        say("graph: replay", i)
        d_stats.zero_()
        _ = ref.float().sum()  # eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got, _ = kb.kb_screen_stats(d_stats, K)
        assert got == want, i


def test_kb_screen_in_a_captured_graph(dev):
    """kb_screen with a caller's workspace, captured and replayed the same
    way: each call leaves the workspace's tickets at zero, so replays need no
    re-initialisation."""
    g = torch.Generator(device=dev).manual_seed(12)
    n, K = 3 * 512 * 67 + 9, 6
    ref = torch.randn(n, generator=g, device=dev)
    cands = [ref + 1e-6 * torch.randn(n, generator=g, device=dev) for _ in range(K)]
    cands[2][n - 1] = float("nan")
    ws = kb.alloc_workspace(K, n, kb.KB_F32, dev)
    d_stats = kb.alloc_stats(K, dev)
    kb.kb_screen(ref, cands, 1e-5, 1e-5, 0, ws, d_stats)
    want, _ = kb.kb_screen_stats(d_stats, K)
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        kb.kb_screen(ref, cands, 1e-5, 1e-5, 0, ws, d_stats)
    torch.cuda.synchronize()
    for i in range(4):
        say("graph kb_screen: replay", i)
        d_stats.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got, _ = kb.kb_screen_stats(d_stats, K)
        assert got == want, i
