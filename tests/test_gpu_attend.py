"""Bare attention core (rs3_attend) through the C ABI against the oracle.

In bf16 the call runs the readout's split-KV attention kernel on a one-frame
bank built from the inputs, so these cases check that kernel on its own:
ragged key tails, several heads and head widths, split counts, the empty and
single-key cases.  Outputs agree with the fp64 oracle within 2e-2 (bf16
inputs, bf16 probabilities, fp32 accumulation) or 1e-4 (fp32)."""
import numpy as np
import pytest

import oracle
from workloads import storage_to_f64, to_storage

pytestmark = pytest.mark.gpu
torch = pytest.importorskip("torch")


def _run(n_q, n_kv, H, d_h, dtype, seed, n_splits=0):
    import paper_2608_22526_amd as rs3
    from paper_2608_22526_amd.session import to_device, to_host
    rng = np.random.default_rng(seed)
    D = H * d_h
    Q, K, V = (to_storage(rng.standard_normal(shape, dtype=np.float32), dtype)
               for shape in ((n_q, D), (max(n_kv, 1), D), (max(n_kv, 1), D)))
    dt = rs3.RS3_BF16 if dtype == "bf16" else rs3.RS3_F32
    ws_bytes = rs3.attend_workspace_size(n_q, n_kv, H, d_h, dt, n_splits)
    ws = torch.zeros(max(ws_bytes, 256), dtype=torch.uint8, device="cuda")
    O = torch.full((n_q, D), float("nan"), dtype=torch.float32, device="cuda")
    rs3.attend(to_device(Q), to_device(K), to_device(V), n_q, n_kv, H, d_h, dt, O, ws, n_splits)
    torch.cuda.synchronize()
    exp = oracle.attend(storage_to_f64(Q, dtype), storage_to_f64(K[:n_kv], dtype), storage_to_f64(V[:n_kv], dtype),
                        H=H)
    return to_host(O).astype(np.float64), exp, storage_to_f64(V[:n_kv], dtype)


@pytest.mark.parametrize("n_q,n_kv,H,d_h", [(300, 1000, 1, 64), (257, 130, 8, 32), (128, 327, 2, 128),
                                            (50, 300, 1, 256), (1, 65, 4, 64)])
def test_attend_bf16_matches_oracle(n_q, n_kv, H, d_h):
    got, exp, _ = _run(n_q, n_kv, H, d_h, "bf16", seed=n_q + n_kv)
    err = np.abs(got - exp).max()
    assert err <= 2e-2, err


def test_attend_split_override_and_degenerate():
    got, exp, _ = _run(200, 777, 2, 64, "bf16", seed=5, n_splits=3)
    assert np.abs(got - exp).max() <= 2e-2
    got, exp, _ = _run(40, 0, 1, 64, "bf16", seed=6)          # no keys: O = 0
    assert np.array_equal(got, np.zeros_like(got))
    got, _, V = _run(40, 1, 1, 64, "bf16", seed=7)            # one key: O = V_1 (bf16 round trip)
    assert np.abs(got - V[0]).max() <= 1e-2


def test_attend_f32_matches_oracle():
    got, exp, _ = _run(37, 150, 2, 32, "f32", seed=8)
    assert np.abs(got - exp).max() <= 1e-4
