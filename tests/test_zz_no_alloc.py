"""a2t_append_attn_noalloc against a2t_append_attn (GPU).

Two caches hold the same stream (config 1's head shape: 32 query / 8 KV
heads, head dim 128, bf16; two layers) filled to ~4,000 resident rows; one
has the default key-split workspace and is driven through a2t_append_attn,
the other is created without a workspace (A2T_FLAG_NO_WORKSPACE) and driven
through a2t_append_attn_noalloc, whose split partials live in the library's
fixed device array.  Two calls in a row (a 22-row unit, then a smaller 3-row
step) must give the same outputs (the bf16 bar, 2e-2; the split plans are the
same, so the outputs are expected to be bit-identical) and the same cache
contents; a call whose partials would not fit the array is rejected with
A2T_ERR_CAPACITY and changes nothing."""
import numpy as np
import pytest

from synth.streams import CONFIGS, make_workload

pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2


def _caches(L, unit_rows, kept_rows, max_step):
    import paper_2609_31224_amd as a2t
    cfg = CONFIGS[1]
    mk = lambda flags: a2t.a2t_cache_create(L, 1, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim,
                                            a2t.A2T_BF16, unit_rows, kept_rows, max_step,
                                            flags=flags, rope_theta=cfg.rope_theta,
                                            attn_scale=cfg.scale)
    return mk(0), mk(a2t.A2T_FLAG_NO_WORKSPACE)


def test_noalloc_matches_append_attn(gpu):
    import torch
    import paper_2609_31224_amd as a2t
    cfg = CONFIGS[1]
    L, Hq, Hkv, D = 2, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    spec = make_workload(cfg, units=200).streams[0]
    fill_units = 182
    max_step = 1024
    ca, cb = _caches(L, 6000, 64, max_step)
    g = torch.Generator(device="cuda")
    g.manual_seed(7)

    def rnd(*shape):
        return torch.randn(shape, generator=g, device="cuda", dtype=torch.float32).to(torch.bfloat16)

    try:
        # identical history in both caches: all-layers appends, no attention
        for st in spec.steps[:fill_units]:
            k, v = rnd(L, st.n, Hkv, D), rnd(L, st.n, Hkv, D)
            for c in (ca, cb):
                a2t.a2t_append(c, a2t.A2T_ALL_LAYERS, [0], [st.n], k, v, st.seg, st.pos, [st.unit])
        R0 = a2t.a2t_stream_info_get(ca, 0)["resident"]
        assert R0 > 3900
        last_pos = int(spec.steps[fill_units - 1].pos[-1])
        steps = [spec.steps[fill_units],   # a 22-row unit
                 None]                     # then a smaller 3-row step
        for call, st in enumerate(steps):
            if st is None:
                seg = np.array([1, 1, 2], np.uint8)
                pos = np.arange(last_pos + 1, last_pos + 4, dtype=np.int32)
                unit, n = spec.steps[fill_units].unit + 1, 3
            else:
                seg, pos, unit, n = st.seg, st.pos, st.unit, st.n
            last_pos = int(pos[-1])
            print(f"[noalloc] call {call + 1}: {n} rows over R={a2t.a2t_stream_info_get(ca, 0)['resident']}",
                  flush=True)
            for layer in range(L):
                k, v, q = rnd(n, Hkv, D), rnd(n, Hkv, D), rnd(n, Hq, D)
                oa, ob = torch.empty_like(q), torch.empty_like(q)
                meta = (seg, pos, [unit]) if layer == 0 else (None, None, None)
                a2t.a2t_append_attn(ca, layer, [0], [n], k, v, *meta, [n], q, oa)
                a2t.a2t_append_attn_noalloc(cb, layer, [0], [n], k, v, *meta, [n], q, ob)
                torch.cuda.synchronize()
                err = float((oa.float() - ob.float()).abs().max())
                assert err <= BF16_TOL, (call, layer, err)
                assert torch.equal(oa, ob), (call, layer, err)
            for c in (ca, cb):
                a2t.a2t_evict(c, [0], [4096], cfg.window)
            for layer in range(L):
                ka, va = a2t.a2t_read_kv(ca, layer, 0)
                kb, vb = a2t.a2t_read_kv(cb, layer, 0)
                assert np.array_equal(ka, kb) and np.array_equal(va, vb)
            assert [a2t.a2t_read_layout(ca, 0)[i].tolist() for i in range(3)] == \
                [a2t.a2t_read_layout(cb, 0)[i].tolist() for i in range(3)]
        # a step whose split partials would exceed the fixed array is refused
        # before anything changes: 1,024 query rows over ~4,000 keys
        n = max_step
        before = a2t.a2t_stream_info_get(cb, 0)
        seg = np.ones(n, np.uint8)
        pos = np.arange(last_pos + 1, last_pos + 1 + n, dtype=np.int32)
        k, v, q = rnd(n, Hkv, D), rnd(n, Hkv, D), rnd(n, Hq, D)
        with pytest.raises(a2t.A2TError) as e:
            a2t.a2t_append_attn_noalloc(cb, 0, [0], [n], k, v, seg, pos, [unit + 1], [n], q,
                                        torch.empty_like(q))
        assert e.value.status == a2t.A2T_ERR_CAPACITY
        assert a2t.a2t_stream_info_get(cb, 0) == before
    finally:
        a2t.a2t_cache_destroy(ca)
        a2t.a2t_cache_destroy(cb)
