"""dwkv_decode_noalloc (the decode with the library's static scratch, for
callers that cannot allocate) against dwkv_decode through the C ABI: two calls
in a row on one GPU, the second on a smaller cache, each equal to
dwkv_decode's output bit for bit and within the benchmark spec's tolerance of the
float64 oracle."""
import numpy as np
import pytest

import oracle
from gpu_util import announce, compare, device_cache, torch_gpu
from synth import LLAMA8B_64K, Workload, generate

pytestmark = pytest.mark.gpu


def test_noalloc_matches_decode_two_calls():
    torch = torch_gpu()
    big = generate(LLAMA8B_64K.with_(context=20000), layers=(0, 4))
    small = generate(Workload(name="noalloc-small", batch=3, n_layers=2, window=2, n_kv_heads=2, n_q_heads=8,
                              head_dim=128, context=700, basis_rank=32, levels=(0, 8, 16),
                              probs=(0.8, 0.15, 0.05), q_dtype="f16", seed=31, ragged=(1, 700)), threads=4)
    for host, layer, pairs in ((big, 2, [(0, 0), (0, 5)]), (small, 1, None)):
        dc = device_cache(host)
        G = host.n_q_heads // host.n_kv_heads
        if pairs is None:
            pairs = [(b, h) for b in range(host.batch) for h in range(host.n_kv_heads)]
        announce(f"decode_noalloc {host.workload.name} layer={layer}")
        got = dc.decode_noalloc(layer).cpu().numpy()
        announce(f"decode {host.workload.name} layer={layer}")
        want = dc.decode(layer).cpu().numpy()
        torch.cuda.synchronize()
        assert np.array_equal(got, want), f"{host.workload.name}: noalloc output differs from dwkv_decode"
        compare(got, oracle.decode(host, layer, heads=pairs), pairs, G, f"noalloc {host.workload.name}")
        del dc


def test_noalloc_with_probe_matches_decode():
    """With an Eq. 3 probe (the wide merge's counters live in the static array
    and are cleared by the reference pass of each call), at one and at three
    positions: outputs and errors equal dwkv_decode's bit for bit, twice in a
    row."""
    torch = torch_gpu()
    from paper_2607_06523_amd import ProbeRef
    from synth.layout import block_values
    host = generate(Workload(name="noalloc-probe", batch=2, n_layers=2, window=2, n_kv_heads=4, n_q_heads=16,
                             head_dim=128, context=1500, basis_rank=48, levels=(0, 4, 8, 16),
                             probs=(0.7, 0.1, 0.1, 0.1), q_dtype="bf16", seed=37, ragged=(2, 1500)), threads=4)
    dc = device_cache(host)
    rng = np.random.default_rng(5)
    T = host.total_tokens
    heads = [3, 1]
    K = rng.standard_normal((2, T, 128)).astype(np.float16)
    V = rng.standard_normal((2, T, 128)).astype(np.float16)
    kd = torch.from_numpy(K.view(np.uint16)).view(torch.float16).cuda()
    vd = torch.from_numpy(block_values(V).view(np.uint16)).view(torch.float16).cuda()
    q_prev = torch.randn((2, host.batch, host.n_q_heads, 128), dtype=torch.float32).to(torch.bfloat16).cuda()
    for name, pr in (("one position", ProbeRef(heads, kd, vd)),
                     ("three positions", ProbeRef(heads, kd, vd, q_prev=q_prev))):
        for rep in range(2):
            announce(f"decode_noalloc with probe, {name}, call {rep}")
            out_n, err_n = dc.decode_noalloc(1, probe=pr)
            out_d, err_d, _ = dc.decode(1, probe=pr)
            torch.cuda.synchronize()
            assert np.array_equal(out_n.cpu().numpy(), out_d.cpu().numpy()), name
            assert np.array_equal(err_n.cpu().numpy(), err_d.cpu().numpy()), name


def test_noalloc_replayed_from_a_graph():
    """The allocation-free decode captured in a HIP graph (it enqueues no
    allocation and no memset) and replayed three times, with eager work and
    synchronizations between the replays: every replay's output equals the
    eager call's bit for bit."""
    torch = torch_gpu()
    host = generate(Workload(name="noalloc-graph", batch=2, n_layers=2, window=2, n_kv_heads=2, n_q_heads=8,
                             head_dim=128, context=3000, basis_rank=48, levels=(0, 4, 8, 16),
                             probs=(0.7, 0.1, 0.1, 0.1), q_dtype="bf16", seed=41, ragged=(1, 3000)), threads=4)
    dc = device_cache(host)
    out = torch.empty((host.batch, host.n_q_heads, 128), dtype=torch.float32, device="cuda")
    announce("decode_noalloc eager")
    want = dc.decode_noalloc(1, out=torch.empty_like(out)).cpu().numpy()
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(side):
        dc.decode_noalloc(1, out=out)                 # warm-up on the capture stream
    torch.cuda.current_stream().wait_stream(side)
    torch.cuda.synchronize()
    graph = torch.cuda.CUDAGraph()
    announce("decode_noalloc graph capture")
    with torch.cuda.graph(graph):
        dc.decode_noalloc(1, out=out)
    for rep in range(3):
        out.fill_(float("nan"))
        announce(f"decode_noalloc graph replay {rep}")
        graph.replay()
        torch.cuda.synchronize()
        assert np.array_equal(out.cpu().numpy(), want), f"replay {rep} differs from the eager call"
        dc.decode(0)                                   # eager work between the replays
        torch.cuda.synchronize()
    del graph
