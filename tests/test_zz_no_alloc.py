"""The allocation-free forward, sp_attn_fwd_static, called through the C ABI
(ctypes, no wrapper allocation): on two calls in a row -- the second with a
smaller problem, so it runs over what the first left in the library's fixed
scratch array -- its outputs equal sp_attn_fwd's (workspace variant, same
kernel and work list) bit for bit, and match the fp64 oracle at the parity
bars."""
import numpy as np
import pytest

import oracle
from tests.helpers import (LSE_MAX_ABS, assert_close, bits_from_dev, from_dev, lib_desc,
                           make_shard, oracle_kw, to_dev)
from workloads import shard_inputs

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def sp():
    import torch
    assert torch.cuda.is_available()
    import paper_2505_22296_amd as m
    m.load()
    return m


def _cases():
    # larger: two packed segments, an empty one and padding rows; 7 real of
    # 8 padded heads at SP 2, rank 1 (slot 3 a dummy), GQA group 7, D = 128
    big = make_shard("noalloc_big", 2100, 2100, 128, 4, 4, 7, 8, 7, 1, 0, [1300, 0, 700],
                     seed_base=4100)
    # smaller: one causal sequence, MHA, D = 64, ragged last tile
    small = make_shard("noalloc_small", 333, 333, 64, 2, 0, 2, 2, 1, 2, 0, [333], seed_base=4200)
    return [big, small]


def test_static_forward_matches_workspace_forward(sp):
    import torch
    lib = sp.load()
    for sh in _cases():
        print(f"{sh.name}: T={sh.T_q} D={sh.D} H_loc={sh.H_loc} real={sh.n_real_loc}", flush=True)
        q, k, v, _ = shard_inputs(sh)
        Q, K, V = (to_dev(x) for x in (q, k, v))
        d = lib_desc(sh)
        o_ref, lse_ref = sp.sp_attn_fwd(d, Q, K, V)
        o = torch.full_like(o_ref, 7.0)
        lse = torch.full_like(lse_ref, float("nan"))
        st = torch.cuda.current_stream().cuda_stream
        rc = lib.sp_attn_fwd_static(d.ref, Q.data_ptr(), K.data_ptr(), V.data_ptr(), o.data_ptr(),
                                    lse.data_ptr(), st)
        assert rc == sp.SP_OK, sp.status_string(rc)
        torch.cuda.synchronize()
        assert np.array_equal(bits_from_dev(o), bits_from_dev(o_ref))
        assert np.array_equal(lse.cpu().numpy().view(np.int32), lse_ref.cpu().numpy().view(np.int32))
        nr = sh.n_real_loc
        RO, RL = oracle.attn_forward(*(oracle.bf16_bits_to_f64(x) for x in (q, k, v)), **oracle_kw(sh))
        assert_close(from_dev(o)[:, :nr], RO[:, :nr], "O")
        fin = np.isfinite(RL[:nr])
        GL = lse.cpu().numpy()[:nr]
        assert np.array_equal(np.isfinite(GL), fin)
        assert np.abs(GL[fin] - RL[:nr][fin]).max() <= LSE_MAX_ABS
        if nr < sh.H_loc:
            assert np.all(bits_from_dev(o)[:, nr:] == 0)
