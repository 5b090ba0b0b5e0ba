"""The tiny workload's re-encode mode end to end on the GPU (2 layers, H = 256, 4/2 heads,
d_h 64, FFN 1024, fp32): the cache is written by the oracle's causal forward over token ids from
the 1000-word vocabulary (keys after rotation, values unrotated; section 5.1, the Text-PRM
re-encode of [x; v]), rounded to its fp32 storage, laid out token by token in pages scattered
over a NaN-filled pool, converted to the stored tile layout by kvprm_pack_kv, and scored by
kvprm_score with the verify token id 999. P(+) and z must equal the re-encode's last position
within the fp32 bar (|dP| <= 1e-5, |dz| <= 4e-5). The mixed variant gives the verify token other
weights than the cached positions (the adapter on the verify token only, section 4.1)."""
import sys

import numpy as np
import pytest
import torch

import synth
from oracle import inputs as oin
from synth.device import DeviceWorkload

from gpu_common import kv

pytestmark = pytest.mark.gpu


def _say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def _token_major_pools(w: synth.Workload, Ks, Vs):
    """[N_L][num_pages][n_kv][16][d] fp32 pools holding candidate b's token t of layer l at
    page page_table[b][t // 16], slot t % 16; every other slot NaN."""
    s = w.shape
    shp = (s.num_layers, w.num_pages, s.num_kv_heads, s.page_size, s.head_dim)
    kt = np.full(shp, np.nan, dtype=np.float32)
    vt = np.full(shp, np.nan, dtype=np.float32)
    for b, L in enumerate(w.lengths):
        for i in range(-(-L // s.page_size)):
            phys = w.page_table[b][i]
            cnt = min(s.page_size, L - i * s.page_size)
            sl = slice(i * s.page_size, i * s.page_size + cnt)
            for l in range(s.num_layers):
                kt[l, phys, :, :cnt] = Ks[b][l][:, sl]
                vt[l, phys, :, :cnt] = Vs[b][l][:, sl]
    return kt, vt


@pytest.mark.parametrize("lengths,mixed", [([512] * 4, False), ([512] * 4, True),
                                           ([512, 301, 16, 0], False)])
def test_reencode_written_cache_scores_like_the_reencode(lengths, mixed):
    _say(f"case: re-encode mode lengths={lengths} mixed={mixed}")
    shape = synth.TINY
    seed = 1000
    r = oin.reencode_batch(shape, seed, lengths, mixed=mixed)
    # device weights: those the verify token runs (theta, or theta' when mixed)
    wseed = seed + synth.ADAPTER_SEED_OFFSET if mixed else seed
    w = synth.make_workload("custom", shape=shape, lengths=lengths, seed=wseed)
    dw = DeviceWorkload(w)
    dw.globals["verify_embed"].copy_(torch.from_numpy(r["verify_embed"].astype(np.float32)))
    kt, vt = _token_major_pools(w, r["K"], r["V"])
    m = kv()
    st = torch.cuda.current_stream().cuda_stream
    ntiles = shape.num_layers * w.num_pages * shape.num_kv_heads
    kp = torch.empty(kt.size, dtype=torch.float32, device="cuda")
    vp = torch.empty(vt.size, dtype=torch.float32, device="cuda")
    ktd, vtd = torch.from_numpy(kt).cuda(), torch.from_numpy(vt).cuda()
    m.kvprm_pack_kv(ktd.data_ptr(), kp.data_ptr(), ntiles, shape.head_dim, "f32", m.KVPRM_KEYS, st)
    m.kvprm_pack_kv(vtd.data_ptr(), vp.data_ptr(), ntiles, shape.head_dim, "f32", m.KVPRM_VALUES,
                    st)
    h = m.kvprm_create(dw.desc(m))
    try:
        batch = dw.batch(m)
        n = m.kvprm_workspace_size(h, batch)
        ws = torch.empty(max(n, 256), dtype=torch.uint8, device="cuda")
        B = len(lengths)
        scores = torch.full((B,), float("nan"), dtype=torch.float32, device="cuda")
        logits = torch.full((B,), float("nan"), dtype=torch.float32, device="cuda")
        m.kvprm_score(h, m.make_cache(kp.data_ptr(), vp.data_ptr(), w.num_pages), batch,
                      dw.readout(m), ws.data_ptr(), n, scores.data_ptr(), logits.data_ptr(), st)
        torch.cuda.synchronize()
    finally:
        m.kvprm_destroy(h)
    p = scores.cpu().numpy().astype(np.float64)
    z = logits.cpu().numpy().astype(np.float64)
    dp, dz = np.max(np.abs(p - r["p"])), np.max(np.abs(z - r["z"]))
    _say(f"  z re-encode {np.round(r['z'], 5)}  max|dP| = {dp:.2e}  max|dz| = {dz:.2e}")
    assert np.all(np.isfinite(p)) and np.all(np.isfinite(z))
    assert dp <= 1e-5 and dz <= 4e-5
