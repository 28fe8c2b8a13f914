"""HIP-graph capture of the library's calls: every entry point enqueues kernels
only (no allocation, no synchronisation, no memset), so a whole step can be
captured once and replayed.  One graph holds a parallel call, a KV append and
the streaming call of the next chunk, a W = 1 ring step, the backward of the
parallel call, and tile gather -> attention over the tile batch -> blend fused
with the one-step update.  It is replayed several times with eager work and
synchronisations in between, and every replay must reproduce the eager
results bit for bit."""
import pytest
import torch

from paper_2609_36757_amd import fastvr
from paper_2609_36757_amd.workloads import make_qkv

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def dev():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fastvr.load()
    return torch.device("cuda:0")


def _run_step(t):
    """Enqueue the whole step on the current stream; outputs go into t's buffers."""
    L = t["L"]
    fastvr.chunk_attn(t["q"], t["k"], t["v"], chunk_len=L, out=t["o"], lse=t["lse"])
    fastvr.kv_cache_append(t["kc"], t["vc"], t["k_new"], t["v_new"], 2 * L)
    fastvr.chunk_attn(t["q_new"], t["kc"], t["vc"], chunk_len=L, q_chunk_offset=2, out=t["so"], lse=t["sl"])
    fastvr.chunk_attn_ring_step(t["q_new"], t["k_new"], t["v_new"], t["rk"], t["rv"], chunk_len=L, chunk_index=2,
                                window_chunks=1, out=t["ro"], lse=t["rl"])
    fastvr.chunk_attn_bwd(t["q"], t["k"], t["v"], t["o"], t["lse"], t["dout"], chunk_len=L, dq=t["dq"], dk=t["dk"],
                          dv=t["dv"], row_stats=t["rs"])
    for x, tl in zip(t["grid"], t["tiles"]):
        fastvr.tile_gather(x, tile=16, overlap=4, out=tl)
    n_t = t["tiles"][0].shape[0] * t["tiles"][0].shape[1]
    tok = lambda x: x.view(n_t, -1, t["H"], t["d"])
    fastvr.chunk_attn(tok(t["tiles"][0]), tok(t["tiles"][1]), tok(t["tiles"][2]), chunk_len=t["tile_chunk"],
                      out=tok(t["to"]), lse=t["tlse"])
    fastvr.tile_blend(t["to"], t["Hg"], t["Wg"], tile=16, overlap=4, z_lq=t["z"], sigma=0.7, out=t["zh"])


def test_graph_replays_match_eager(dev):
    B, H, d, L = 1, 2, 128, 200
    print("\n[gpu case] graph capture: parallel, append + stream, ring step, backward, tiles", flush=True)
    q, k, v = (x.to(dev) for x in make_qkv(B, 3 * L, 3 * L, H, d, 71))
    g = torch.Generator().manual_seed(72)
    t = {"L": L, "H": H, "d": d, "q": q, "k": k, "v": v}
    t["o"] = torch.empty((B, 3 * L, H, d), dtype=torch.float32, device=dev)
    t["lse"] = torch.empty((B, H, 3 * L), dtype=torch.float32, device=dev)
    t["kc"] = torch.zeros((B, 3 * L, H, d), dtype=torch.bfloat16, device=dev)
    t["vc"] = torch.zeros_like(t["kc"])
    t["kc"][:, :2 * L].copy_(k[:, :2 * L])
    t["vc"][:, :2 * L].copy_(v[:, :2 * L])
    t["q_new"], t["k_new"], t["v_new"] = (x[:, 2 * L:].contiguous() for x in (q, k, v))
    t["so"] = torch.empty((B, L, H, d), dtype=torch.float32, device=dev)
    t["sl"] = torch.empty((B, H, L), dtype=torch.float32, device=dev)
    t["rk"] = torch.zeros((B, 2 * L, H, d), dtype=torch.bfloat16, device=dev)
    t["rv"] = torch.zeros_like(t["rk"])
    t["rk"][:, L:].copy_(k[:, L:2 * L])   # chunk 1 in slot 1
    t["rv"][:, L:].copy_(v[:, L:2 * L])
    t["ro"] = torch.empty((B, L, H, d), dtype=torch.float32, device=dev)
    t["rl"] = torch.empty((B, H, L), dtype=torch.float32, device=dev)
    t["dout"] = torch.randn((B, 3 * L, H, d), generator=g).to(torch.bfloat16).to(dev)
    t["dq"] = torch.empty((B, 3 * L, H, d), dtype=torch.float32, device=dev)
    t["dk"], t["dv"] = torch.empty_like(t["dq"]), torch.empty_like(t["dq"])
    t["rs"] = torch.empty((B, H, 2, 3 * L), dtype=torch.float32, device=dev)
    T, Hg, Wg = 2, 20, 28
    t["Hg"], t["Wg"] = Hg, Wg
    t["grid"] = [torch.randn((B, T, Hg, Wg, H * d), generator=g).to(torch.bfloat16).to(dev) for _ in range(3)]
    ny, Ly = fastvr.tile_axis(Hg, 16, 4)
    nx, Lx = fastvr.tile_axis(Wg, 16, 4)
    t["tiles"] = [torch.empty((B, ny * nx, T, Ly, Lx, H * d), dtype=torch.bfloat16, device=dev) for _ in range(3)]
    t["tile_chunk"] = Ly * Lx
    t["to"] = torch.empty((B, ny * nx, T, Ly, Lx, H * d), dtype=torch.float32, device=dev)
    t["tlse"] = torch.empty((B * ny * nx, H, T * Ly * Lx), dtype=torch.float32, device=dev)
    t["z"] = torch.randn((B, T, Hg, Wg, H * d), generator=g).to(torch.bfloat16).to(dev)
    t["zh"] = torch.empty((B, T, Hg, Wg, H * d), dtype=torch.float32, device=dev)
    outs = ["o", "lse", "kc", "vc", "so", "sl", "rk", "rv", "ro", "rl", "dq", "dk", "dv", "rs", "to", "tlse", "zh"]

    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        _run_step(t)   # eager, on the stream the graph is captured from
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    eager = {n: t[n].clone() for n in outs}
    eager["tiles"] = [x.clone() for x in t["tiles"]]

    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        _run_step(t)
    torch.cuda.synchronize()
    for rep in range(3):
        for n in ("o", "lse", "so", "sl", "ro", "rl", "dq", "dk", "dv", "rs", "to", "tlse", "zh"):
            t[n].fill_(float("nan"))
        for x in t["tiles"]:
            x.zero_()
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for n in outs:
            assert torch.equal(t[n], eager[n]), (rep, n)
        for x, e in zip(t["tiles"], eager["tiles"]):
            assert torch.equal(x, e), (rep, "tiles")
    print("[parity] graph replays x3 bit-identical to eager", flush=True)
