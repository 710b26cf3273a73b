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
