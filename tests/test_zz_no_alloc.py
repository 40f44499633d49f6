"""The key encoder's entry point for callers that cannot allocate
(pf_key_encode_static: the projection's fp64 work batch in a static device
buffer of the library) against pf_key_encode (the projection's own work
buffer): identical keys, on two calls in a row with the second smaller, on
fp32 and bf16 states, through the C ABI."""
import numpy as np
import pytest

import oracle
import synth
import keycheck

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def pf():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    import paper_2609_32166_amd as pf
    pf.lib()
    return pf


@pytest.mark.parametrize("H,dtype,n1,n2", [(2048, "bf16", 150, 17), (256, "f32", 70, 3),
                                           (3584, "bf16", 64, 1)])
def test_static_encode_equals_allocating_encode(pf, H, dtype, n1, n2):
    import torch
    R = synth.key_projection(H, 91)
    kp = pf.pf_keyproj_create(R)
    R64 = R.astype(np.float64)
    for call, n in enumerate((n1, n2)):
        h = synth.hidden_states(n, H, 92 + call)
        t = torch.from_numpy(np.ascontiguousarray(h, np.float32)).cuda()
        if dtype == "bf16":
            t = t.to(torch.bfloat16)
        k_alloc = torch.full((n, pf.KEY_DIM), 55, dtype=torch.int8, device="cuda")
        k_static = torch.full((n, pf.KEY_DIM), -55, dtype=torch.int8, device="cuda")
        pf.pf_key_encode(kp, t, k_alloc)
        pf.pf_key_encode_static(kp, t, k_static)
        torch.cuda.synchronize()
        a, b = k_alloc.cpu().numpy(), k_static.cpu().numpy()
        print(f"H={H} {dtype} call {call}: {n} rows, identical={bool((a == b).all())}")
        assert (a == b).all(), np.argwhere(a != b)[:8]
        hv = t.to(torch.float64).cpu().numpy()
        keycheck.check_codes(b, R64, hv, oracle.key_project(R64, hv))
