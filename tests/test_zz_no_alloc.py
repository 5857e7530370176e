"""tvq_attention_decode_noalloc (attention with the library's static scratch in place of a
caller's workspace), through the C ABI, against tvq_attention_decode with a workspace: the
same kernels and chunk plan, so the outputs must be identical bit for bit, on two calls in a
row (the second smaller, so it reads partials the first call left behind only if it failed to
write its own), and within the oracle's attention bar.  A call whose partials exceed the
scratch is refused before any launch."""
import sys

import numpy as np
import pytest

import oracle
import workloads
from workloads import LayerCfg

from parity import Setup, attention_error_bar, bf16_bits_to_torch, torch_to_np

pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def _case(d, B, H, T, seed):
    import torch
    w = workloads.get("C2")
    table = [LayerCfg(64, 64), LayerCfg(256, 256)]
    s = Setup(2, H, d, table, workloads.sign_table(seed, 2, d)).build()
    ww = workloads.Workload(w.name, 2, B, H, T, d, "bf16", table, seed, w.sign_seed, w.k_dist,
                            w.v_dist, w.n_outlier, w.outlier_scale)
    k, v = workloads.generate(ww, "K"), workloads.generate(ww, "V")
    lay = s.gpu.layout(B, T)
    cache = torch.zeros((lay.total_bytes,), dtype=torch.uint8, device="cuda")
    s.gpu.encode(bf16_bits_to_torch(k).cuda(), bf16_bits_to_torch(v).cuda(), cache, lay)
    torch.cuda.synchronize()
    return s, lay, cache


@pytest.mark.parametrize("d", [128, 64])
def test_noalloc_attention_matches_the_workspace_entry_point(gpu, d):
    import torch
    import paper_2603_27467_amd as tvq
    H, G = 2, 4
    s, lay, cache = _case(d, 3, H, 1500, seed=31)
    rng = np.random.default_rng(32)
    host = torch_to_np(cache)
    # two calls in a row, the second over fewer tokens, fewer sequences' worth of work and the
    # other layer; each against the workspace entry point and the oracle
    for layer, t_end, o_dtype in ((1, 1500, torch.float32), (0, 333, torch.bfloat16)):
        q = torch.from_numpy(rng.standard_normal((3, H * G, d)).astype(np.float32)).cuda()
        ref = torch.full((3, H * G, d), float("nan"), dtype=o_dtype, device="cuda")
        got = torch.full_like(ref, float("nan"))
        scale = 1.0 / np.sqrt(d)
        s.gpu.attention(cache, lay, layer, t_end, q, ref, scale)
        s.gpu.attention_noalloc(cache, lay, layer, t_end, q, got, scale)
        torch.cuda.synchronize()
        need = s.gpu.attention_workspace_bytes(3, H * G, t_end)
        same = torch.equal(ref.view(torch.int16 if o_dtype == torch.bfloat16 else torch.int32),
                           got.view(torch.int16 if o_dtype == torch.bfloat16 else torch.int32))
        q64 = q.cpu().numpy().astype(np.float64)
        want = s.orc.attention_decode(host, 3, lay.capacity_tokens, layer, t_end, q64, scale)
        bar = attention_error_bar(s, host, 3, lay.capacity_tokens, layer, t_end, q64, scale,
                                  want, o_dtype == torch.float32)
        err = np.linalg.norm(got.float().cpu().numpy().astype(np.float64) - want, axis=-1)
        _say(f"[noalloc d={d} layer={layer} t_end={t_end} {o_dtype}] partials {need} bytes of "
             f"{tvq.TVQ_ATTENTION_SCRATCH_BYTES}; identical to the workspace call: {same}; "
             f"max |err|/bar vs oracle {(err / bar).max():.3f}")
        assert same
        assert (err <= bar).all()


def test_noalloc_attention_refuses_more_than_its_scratch(gpu):
    """48 sequences x 64 query heads over 65536 tokens need ~26 MB of partials: refused with
    TVQ_ERR_SCRATCH before anything is launched (the output keeps its fill)."""
    import torch
    import paper_2603_27467_amd as tvq
    d, H, G, B, T = 128, 2, 32, 48, 65536
    s = Setup(1, H, d, [LayerCfg(64, 64)], workloads.sign_table(3, 1, d)).build()
    lay = s.gpu.layout(B, T)
    need = s.gpu.attention_workspace_bytes(B, H * G, T)
    assert need > tvq.TVQ_ATTENTION_SCRATCH_BYTES
    cache = torch.zeros((lay.total_bytes,), dtype=torch.uint8, device="cuda")
    q = torch.zeros((B, H * G, d), dtype=torch.float32, device="cuda")
    out = torch.full_like(q, 7.0)
    with pytest.raises(tvq.TvqError) as e:
        s.gpu.attention_noalloc(cache, lay, 0, T, q, out, 0.1)
    assert e.value.status == tvq.TVQ_ERR_SCRATCH
    torch.cuda.synchronize()
    assert bool((out == 7.0).all())
    _say(f"[noalloc] {need} bytes of partials refused ({tvq.TVQ_ATTENTION_SCRATCH_BYTES} held)")
