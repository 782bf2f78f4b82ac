"""The decode entry point that allocates nothing (mosaic_decode_attention_noalloc,
for callers that cannot allocate device memory): called through the C ABI, its
output must equal mosaic_decode_attention's on the same cache, for two calls in
a row on the one GPU buffer, the second with a smaller cache."""
import ctypes as C
import math

import numpy as np
import pytest
import torch

from _parity import gpu_cache, params_pair
from workloads import gen

pytestmark = pytest.mark.gpu


def _noalloc(cache, q, scale):
    out = torch.empty((cache.num_seqs, cache.params.num_kv_heads * cache.params.group_size, 128),
                      dtype=torch.float32, device=cache.device)
    st = cache.lib.mosaic_decode_attention_noalloc(cache._h, C.c_void_p(q.data_ptr()), C.c_void_p(out.data_ptr()),
                                                   C.c_float(scale),
                                                   C.c_void_p(torch.cuda.current_stream().cuda_stream))
    assert st == 0, cache.lib.mosaic_last_error().decode()
    return out


def test_noalloc_decode_equals_workspace_decode_twice():
    scale = 1.0 / math.sqrt(128)
    runs = [gen.spec("c3", ctx=(3000, 2100, 1300), hkv=4, kind="gauss"),   # larger first
            gen.spec("c1", ctx=(700,), hkv=2)]                               # then smaller
    for i, spec in enumerate(runs):
        print(f"[noalloc] call {i}: ctx={spec.ctx} hkv={spec.hkv} {spec.dtype}", flush=True)
        cap = spec.max_ctx + 64
        lay = gen.make_layer(spec, 0, capacity=cap)
        lp, _ = params_pair(spec)
        cache = gpu_cache(lp, spec, lay, cap)
        q = gen.make_queries(spec, i).cuda()
        want = cache.decode(q, scale).clone()
        got = _noalloc(cache, q, scale)
        torch.cuda.synchronize()
        assert torch.equal(got, want), f"call {i}: max diff {(got - want).abs().max().item():.3e}"
        # and again: the buffer keeps the last call's contents, which nothing reads
        got2 = _noalloc(cache, q, scale)
        torch.cuda.synchronize()
        assert torch.equal(got2, want)
