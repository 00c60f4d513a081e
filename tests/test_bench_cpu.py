"""Host logic of bench.py that needs no GPU: the gradient comparison used for
the bit-identity claims (element by element, or per-chunk hashes where a
snapshot cannot hold a copy) and the LDS-kernel rule mirrored from the
library."""
import os
import sys

import pytest

torch = pytest.importorskip("torch")
sys.path.insert(0, os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
import bench  # noqa: E402


def test_hash_detects_every_single_differing_element():
    t = torch.randn(3 * 1000 + 7)
    d = bench._digest(t)
    assert d == bench._digest(t.clone())
    for i in (0, 1, 1234, t.numel() - 1):
        u = t.clone()
        u.view(torch.int32)[i] ^= 1          # one bit of one element
        assert bench._digest(u) != d, i
    # NaNs compare by their bit patterns
    n1 = torch.full((4,), float("nan"))
    n2 = n1.clone()
    n2.view(torch.int32)[2] ^= 1
    assert bench._digest(n1) != bench._digest(n2)


def test_hash_chunks_cover_the_whole_tensor(monkeypatch):
    monkeypatch.setattr(bench, "_HASH_CHUNK", 16)
    t = torch.randn(16 * 3 + 5)
    d = bench._digest(t)
    assert d[0] == "hash64" and d[1] == t.numel() and len(d[2]) == 4
    u = t.clone()
    u.view(torch.int32)[-1] ^= 1            # the last, partial chunk
    assert bench._digest(u)[2][:3] == d[2][:3] and bench._digest(u)[2][3] != d[2][3]


def test_same_gradients_mixes_copies_and_hashes():
    a = {"dW": torch.randn(40), "db": torch.randn(5), "loss": 1.5}
    b = {k: (v.clone() if hasattr(v, "clone") else v) for k, v in a.items()}
    assert bench.same_gradients(a, b)
    h = dict(a, dW=bench._digest(a["dW"]))
    assert bench.same_gradients(h, b) and bench.same_gradients(b, h)
    b["dW"].view(torch.int32)[7] ^= 1
    assert not bench.same_gradients(h, b)
    assert not bench.same_gradients(a, dict(a, loss=1.25))
    assert bench.comparison_kind(h).startswith("64-bit hash per 256 MiB chunk for dW")
    assert bench.comparison_kind(a) == "element by element"


def test_lds_rule_of_the_4096_lstm():
    import synth
    import paper_1806_01117_amd as amb
    spec = amb.ProblemSpec.from_workload(synth.get("lstm_h4096_t20000"))
    assert bench.lds_kernels(spec, []) == (True, True)
    assert bench.lds_kernels(spec, [("lds_gemm", 0)]) == (False, False)
    small = amb.ProblemSpec.from_workload(synth.get("lstm_h512_t1000"))
    assert bench.lds_kernels(small, []) == (False, False)


def test_prod_split_rule():
    import synth
    import paper_1806_01117_amd as amb
    big = amb.ProblemSpec.from_workload(synth.get("lstm_h4096_t20000"))
    assert bench.prod_split_parts(big, []) == 4                     # 128 tiles of 128 x 128, 256 stages
    assert bench.prod_split_parts(big, [("prod_split", 0)]) == 1
    assert bench.prod_split_parts(big, [("lds_gemm", 0)]) == 1
    ragged = amb.ProblemSpec.from_workload(synth.get("lstm_h4096_t20000").with_(batch=300, input=96, hidden=1024))
    assert bench.prod_split_parts(ragged, [("lds_gemm", 2)]) == 4   # 24 tiles, 64 stages: 4 parts of 16
    rnn = amb.ProblemSpec.from_workload(synth.get("lstm_h4096_t20000").with_(cell="rnn", batch=300, input=64,
                                                                            hidden=1024))
    assert bench.prod_split_parts(rnn, [("lds_gemm", 2)]) == 1      # 16 stages: a part would hold 8


def test_mlp_layer_work_reduces_to_one_width():
    B, w, n = 8, 32, 5
    f, b = bench.mlp_layer_work([w] * (n + 1), B)
    assert set(f) == {"fwd", "adj", "dw"}
    assert f["fwd"] == 2.0 * B * w * w
    # the adjoint also forms zbar_{l+1} W_{l+1}, for every layer but the last
    assert f["adj"] == 2.0 * B * w * w * (1 + (n - 1) / n)
    assert f["dw"] == 2.0 * B * w * (w + 1)
    assert b["fwd"] == 4.0 * (w * w + w + 2 * B * w)
    # widths that alternate: the mean over layers of each class
    f2, _ = bench.mlp_layer_work([16, 32, 16], 4)
    assert f2["fwd"] == (2 * 4 * 16 * 32 + 2 * 4 * 32 * 16) / 2
    assert f2["adj"] == (2 * 4 * 16 * 32 + 2 * 4 * 32 * 16 + 2 * 4 * 32 * 16) / 2


def test_pmc_table_names_kernel_instances():
    from paper_1806_01117_amd.pmc_summary import _instance
    assert _instance("void ambptt::(anonymous namespace)::mlpv_gemm<3, 1, 4>(ambptt::MlpvArgs)") == "mlpv_gemm<3, 1, 4>"
    assert _instance("ambptt::(anonymous namespace)::dw_f32_big(ambptt::DwArgs)") == "dw_f32_big"
    assert _instance("void ambptt::(anonymous namespace)::mlpv_dw<1>(ambptt::(anonymous namespace)::MlpvDwGroup)") \
        == "mlpv_dw<1>"
    assert _instance("__amd_rocclr_copyBuffer") == "__amd_rocclr_copyBuffer"
