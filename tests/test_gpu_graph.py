"""HIP-graph capture of the whole path: replays must equal eager execution.

The benchmark times one step (window-start quantization, every decode launch
and the window commits) as a captured graph.  Here the same sequence is run
eagerly and captured; the graph is replayed several times with unrelated eager
work and synchronisations in between, and every replay must reproduce the eager
outputs and final state bit for bit (all kernels use fixed reduction orders).
"""
import pytest
import torch

from paper_2609_38166_amd import binding as B
from paper_2609_38166_amd import synth

pytestmark = pytest.mark.gpu

CASES = {
    # KDA, 2.5 windows (a partial window left open), int8
    "kda": dict(batch=2, heads_v=4, heads_k=4, window=8, n_comp=4, gate=synth.GATE_DIAG, code=synth.CODE_INT8,
                steps=20),
    # GDN with grouped keys, e4m3 codes
    "gdn_gqa_e4m3": dict(batch=2, heads_v=4, heads_k=2, window=8, n_comp=2, gate=synth.GATE_SCALAR,
                         code=synth.CODE_E4M3, steps=20),
}


def _inputs(c, seed):
    g = torch.Generator(device="cuda")
    g.manual_seed(seed)
    B_, Hv, Hk, T = c["batch"], c["heads_v"], c["heads_k"], c["steps"]
    S0 = torch.randn((B_, Hv, 128, 128), device="cuda", generator=g) * 0.05
    q = torch.randn((T, B_, Hk, 128), device="cuda", generator=g)
    k = torch.randn((T, B_, Hk, 128), device="cuda", generator=g)
    q /= q.norm(dim=-1, keepdim=True)
    k /= k.norm(dim=-1, keepdim=True)
    v = torch.randn((T, B_, Hv, 128), device="cuda", generator=g)
    ash = (T, B_, Hv, 128) if c["gate"] == synth.GATE_DIAG else (T, B_, Hv)
    a = torch.rand(ash, device="cuda", generator=g) * 0.4 + 0.6
    b = torch.rand((T, B_, Hv), device="cuda", generator=g)
    return S0, q, k, v, a, b


def _run(dims, st, c, S0, toks, outs):
    """quantize, then every decode step (each into its own output) and the commits."""
    q, k, v, a, b = toks
    B.leapquant_quantize_state(dims, S0, st)
    for t in range(c["steps"]):
        B.leapquant_decode_step(dims, st, q[t], k[t], v[t], a[t], b[t], outs[t])
        if (t + 1) % c["window"] == 0:
            B.leapquant_window_commit(dims, st)


def _snapshot(st):
    return {f: getattr(st, f).clone() for f in B.FIELDS}


@pytest.mark.parametrize("name", sorted(CASES))
def test_graph_replays_equal_eager(name):
    c = CASES[name]
    dims = B.make_dims(c["batch"], c["heads_v"], c["heads_k"], window=c["window"], n_comp=c["n_comp"],
                       power_iters=4, gate=c["gate"], code=c["code"])
    S0, *toks = _inputs(c, 1234)
    shape_o = (c["batch"], c["heads_v"], 128)

    st_e = B.State.empty(dims)
    out_e = [torch.empty(shape_o, device="cuda") for _ in range(c["steps"])]
    _run(dims, st_e, c, S0, toks, out_e)
    torch.cuda.synchronize()
    ref_state = _snapshot(st_e)
    ref_out = torch.stack(out_e)
    assert torch.isfinite(ref_out).all()

    st_g = B.State.empty(dims)
    out_g = [torch.empty(shape_o, device="cuda") for _ in range(c["steps"])]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):                   # warm-up pass on the capture stream
        _run(dims, st_g, c, S0, toks, out_g)
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        _run(dims, st_g, c, S0, toks, out_g)
    torch.cuda.synchronize()

    scratch = torch.randn((8, 1 << 16), device="cuda")
    for rep in range(3):
        for o in out_g:
            o.fill_(float("nan"))
        st_g.rec_len.fill_(7)                       # the replay's quantization must reset it
        scratch.mul_(1.0001).add_(0.5)              # unrelated eager work between replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        got = torch.stack(out_g)
        assert torch.equal(got, ref_out), f"{name}: replay {rep} outputs differ from eager"
        for f, ref in ref_state.items():
            assert torch.equal(getattr(st_g, f), ref), f"{name}: replay {rep} state field {f} differs"
    assert B.leapquant_check_error(st_g) == 0
