"""The seeded input generators: shapes, dtypes, determinism and the structure
each workload promises (CPU, reduced vocabulary)."""
import torch

from paper_2405_19261_amd import workloads as W


def test_workload_table():
    assert [W.WORKLOADS[c].B for c in range(1, 6)] == [1, 8, 32, 128, 256]
    assert W.WORKLOADS[3].logit_bytes() == 262_144_000
    assert W.WORKLOADS[4].greedy and not W.WORKLOADS[3].greedy


def test_shapes_dtypes_and_determinism():
    for cfg in range(1, 6):
        wl = W.WORKLOADS[cfg].with_(V=min(W.WORKLOADS[cfg].V, 1536), B=min(W.WORKLOADS[cfg].B, 8))
        a = W.generate(wl, 3)
        b = W.generate(wl, 3)
        c = W.generate(wl, 4)
        G = wl.gamma + 1
        assert a["q"].shape == (wl.B, G, wl.V) and a["p"].shape == (wl.B, G, wl.V)
        assert a["q"].dtype == (torch.float32 if wl.dtype == "f32" else torch.bfloat16)
        assert a["draft"].shape == (wl.B, wl.gamma) and a["draft"].dtype == torch.int32
        assert a["uniforms"].shape == (wl.B, G)
        assert ((a["uniforms"] >= 0) & (a["uniforms"] < 1)).all()
        assert ((a["draft"] >= 0) & (a["draft"] < wl.V)).all()
        for k in a:
            assert torch.equal(a[k], b[k]), k
        assert not torch.equal(a["q"], c["q"])


def test_greedy_drafts_are_first_argmax():
    wl = W.WORKLOADS[4].with_(V=1024, B=6)
    a = W.generate(wl, 0)
    ref = torch.argmax(a["q"][:, :wl.gamma].float(), -1).to(torch.int32)
    assert torch.equal(a["draft"], ref)
    assert (a["temperature"] == 0).all()


def test_stress_mix_structure():
    wl = W.WORKLOADS[5].with_(V=1024, B=16)
    a = W.generate(wl, 0)
    same = [(a["q"][b] == a["p"][b]).all().item() for b in range(wl.B)]
    assert sum(same) == wl.B // 4
    assert set(a["temperature"].tolist()) <= {0.5, 0.699999988079071, 1.0}
    pairs = {(int(r), round(float(al), 4)) for r, al in zip(a["rule"], a["alpha"])}
    assert pairs <= {(0, 0.4), (1, 0.05), (2, 0.1)}


def test_zipf_rows_are_permuted_ranks():
    g = torch.Generator().manual_seed(0)
    z = W._zipf_rows(3, 500, 1.2, g, "cpu")
    ref = torch.sort(-1.2 * torch.log(torch.arange(1, 501, dtype=torch.float64)).float())[0]
    for r in range(3):
        assert torch.equal(torch.sort(z[r])[0], torch.sort(z[0])[0])
        torch.testing.assert_close(torch.sort(z[r])[0], ref, rtol=0, atol=2e-6)
    assert not torch.equal(z[0], z[1])
