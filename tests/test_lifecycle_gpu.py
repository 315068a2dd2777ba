"""One batch through the whole path on one cache, through the C ABI: chunked prefill over the compressed history
(§2.2.1), the chunk's compression into the reserved ragged pages (§4.1, Eq. 4), chunk after chunk, then decode
steps on one open-ended plan with the step's token appended inside the decode launch (§2.2.3, §4.2, §4.3).
Every stage is checked against the oracle run on its own copy of the cache."""
import dataclasses

import numpy as np
import pytest
import torch

import oracle
from gpu_helpers import check_close, say
from workloads import Geometry, custom

pytestmark = pytest.mark.gpu

if torch.cuda.is_available():
    from paper_2606_06302_amd import tangram as tg
    from paper_2606_06302_amd.runner import CompressSession, DecodeSession, PrefillSession, Tables


def _f64(t):
    return t.float().cpu().numpy().astype(np.float64)


@pytest.mark.parametrize("geom,C,n_chunks", [(Geometry(1, 8, 32, 128, 16, 2), 256, 3),
                                             (Geometry(1, 4, 20, 128, 16, 4), 200, 2)])
def test_prefill_compress_decode_lifecycle(geom, C, n_chunks):
    """Chunk c attends over the entries the earlier chunks kept plus its own keys (bf16 tolerance against the
    oracle over every row), then keeps Top(count) of its entries in the pages (the whole pool bit-exact against
    the oracle's); the chunks fill each head's reservation exactly.  Decode steps then append every step's
    token inside the decode launch and attend over the grown cache (outputs within the bf16 tolerance, the
    pool bit-exact, the live lengths exact)."""
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    g = geom
    B, T, seed = 3, 5, 2400 + C
    wl = custom(seed, g, B, "bf16", np.full(B, n_chunks * C), chunk_len=C)
    t = Tables(wl, headroom=np.full(B, T, dtype=np.int32))
    shape = (t.pool_pages, 2, g.heads_per_group, g.page_size, g.head_dim)
    pool = torch.zeros(shape, dtype=torch.bfloat16, device="cuda")
    ref_pool = np.zeros(shape)
    tab = dict(offsets=t.pt_offsets, pages=t.pt_pages, group_of=t.group_of, slot_of=t.slot_of)
    hist = np.zeros((B, 1, g.num_kv_heads), dtype=np.int32)
    for c in range(n_chunks):
        wc = dataclasses.replace(wl, seed=seed + 1 + c)   # the chunk's own queries, keys, values and scores
        ps = PrefillSession(wc, tables=t, fill="host", pool=pool, hist_len=hist)
        ps.run()
        torch.cuda.synchronize()
        ref = oracle.prefill_attention(_f64(ps.q), _f64(ps.k_new), _f64(ps.v_new), ref_pool, 0, geom=g,
                                       kv_len=hist, **tab)
        err = check_close(_f64(ps.out).reshape(-1, g.head_dim), ref.reshape(-1, g.head_dim), "bf16",
                          f"prefill chunk {c}")
        starts, toks = np.full(B, c * C, dtype=np.int32), np.full(B, C, dtype=np.int32)
        cs = CompressSession(wc, t, pool, starts, toks, k_new=ps.k_new, v_new=ps.v_new)
        cs.run()
        torch.cuda.synchronize()
        ref_pool, _, cur, cnt = oracle.compress_chunk(_f64(ps.k_new), _f64(ps.v_new), cs.scores.cpu().numpy(),
                                                      ref_pool, 0, geom=g, ratio=wl.ratio, capacity=t.kv_len,
                                                      chunk_start=starts, chunk_tokens=toks, **tab)
        assert np.array_equal(cur.reshape(hist.shape), hist), f"chunk {c}: write cursors"
        assert np.array_equal(_f64(pool), ref_pool), f"chunk {c}: pool differs after compression"
        hist = (cur + cnt).reshape(hist.shape).astype(np.int32)
        say(f"lifecycle {g} chunk {c}: prefill max abs {err[0]:.2e}, {int(cnt.sum())} rows kept")
    assert np.array_equal(hist, t.kv_len), "the chunks fill each head's reservation exactly"

    s = DecodeSession(wl, tables=t, mode=tg.TG_PLAN_AOT_FILL, n_bins=64, split_target=128, fill="host",
                      pool=pool.view(-1), open_end=True)
    s.enable_append(fused=True)
    rng = np.random.default_rng(seed)
    live = t.kv_len.copy()
    tok_shape = (g.num_layers, B, g.num_kv_heads, g.head_dim)
    for step in range(1, T + 1):
        k = torch.from_numpy(rng.standard_normal(tok_shape, dtype=np.float32)).to(torch.bfloat16)
        v = torch.from_numpy(rng.standard_normal(tok_shape, dtype=np.float32)).to(torch.bfloat16)
        q = torch.from_numpy(rng.standard_normal(tuple(s.q.shape), dtype=np.float32)).to(torch.bfloat16)
        s.k_tok.copy_(k.cuda())
        s.v_tok.copy_(v.cuda())
        s.q.copy_(q.cuda())
        s.run_decode_step()
        torch.cuda.synchronize()
        ref_pool, live, full = oracle.append_token(_f64(k)[0], _f64(v)[0], ref_pool, 0, geom=g, live_len=live, **tab)
        assert full == []
        assert np.array_equal(s.live_len.cpu().numpy(), live), f"step {step}: live lengths"
        assert np.array_equal(_f64(s.pool).reshape(shape), ref_pool), f"step {step}: pool"
        O, _ = oracle.decode_attention(_f64(q)[0], ref_pool, 0, geom=g, batch=B, kv_len=live, **tab)
        check_close(_f64(s.out[0]).reshape(-1, g.head_dim), O.reshape(-1, g.head_dim), "bf16", f"decode step {step}")
    assert int(s.full.item()) == 0
