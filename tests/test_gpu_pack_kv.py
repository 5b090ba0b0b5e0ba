"""kvprm_pack_kv on the GPU: token-major cache tiles -> the stored K and V tile layouts, checked
bit for bit by decoding every packed tile back with the oracle's layout decoders
(kvprm_oracle.k_tile_to_tokens / v_tile_to_tokens, pinned on the CPU against the layout
formulas), for every cache dtype and head size; bytes past the destination stay untouched."""
import sys

import numpy as np
import pytest
import torch

from oracle import kvprm_oracle as ko

from gpu_common import kv

pytestmark = pytest.mark.gpu

_UINT = {1: np.uint8, 2: np.uint16, 4: np.uint32}


@pytest.mark.parametrize("dtype,eb", [("f32", 4), ("bf16", 2), ("fp8", 1)])
@pytest.mark.parametrize("d", [64, 128])
def test_pack_kv_roundtrip_bitwise(dtype, eb, d):
    print(f"case: pack_kv {dtype} d={d}", flush=True)
    sys.stdout.flush()
    m = kv()
    ntiles = 37
    n = ntiles * 16 * d * eb
    rng = np.random.default_rng(d * 10 + eb)
    host = rng.integers(0, 256, size=n, dtype=np.uint8)
    src = torch.from_numpy(host).cuda()
    guard = 4096
    st = torch.cuda.current_stream().cuda_stream
    for part, dec in ((m.KVPRM_KEYS, ko.k_tile_to_tokens), (m.KVPRM_VALUES, ko.v_tile_to_tokens)):
        dst = torch.full((n + guard,), 0xA5, dtype=torch.uint8, device="cuda")
        m.kvprm_pack_kv(src.data_ptr(), dst.data_ptr(), ntiles, d, dtype, part, st)
        torch.cuda.synchronize()
        out = dst.cpu().numpy()
        assert np.all(out[n:] == 0xA5)
        packed = out[:n].view(_UINT[eb]).reshape(ntiles, 16 * d)
        tok = host.view(_UINT[eb]).reshape(ntiles, 16, d)
        for t in range(ntiles):
            assert np.array_equal(dec(packed[t], 16, d, eb), tok[t]), (part, t)
    # nothing to do for zero tiles (null pointers accepted)
    m.kvprm_pack_kv(0, 0, 0, d, dtype, m.KVPRM_KEYS, st)
