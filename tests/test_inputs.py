"""The seeded input generators: host (C) and torch implementations agree bitwise, page
placement is a bijection, and the workload mixes follow their stated distributions."""
import numpy as np
import pytest
import torch

import wisp_inputs as wi


@pytest.mark.parametrize("dtype", [torch.bfloat16, torch.float32])
def test_host_and_torch_generators_agree(dtype):
    wi._FORCE_TORCH_GEN = False
    a = wi.normal_tensor(5, "x", (3, 1000), 0.02, dtype)
    wi._FORCE_TORCH_GEN = True
    try:
        b = wi.normal_tensor(5, "x", (3, 1000), 0.02, dtype)
        k1, v1 = wi.kv_values(7, 2, 3, 5, 40, 8, 128, "cpu", dtype)
    finally:
        wi._FORCE_TORCH_GEN = False
    k2, v2 = wi.kv_values(7, 2, 3, 5, 40, 8, 128, "cpu", dtype)
    iv = torch.int16 if dtype == torch.bfloat16 else torch.int32
    assert torch.equal(a.view(iv), b.view(iv))
    assert torch.equal(k1.view(iv), k2.view(iv)) and torch.equal(v1.view(iv), v2.view(iv))


def test_generator_statistics_and_slices():
    w = wi.normal_tensor(1, "stats", (1 << 20,), 0.02, torch.float32).double()
    assert abs(w.mean().item()) < 1e-4 and abs(w.std().item() - 0.02) < 2e-4
    # a slice of the stream regenerates on its own
    k_all, _ = wi.kv_values(3, 0, 1, 0, 50, 2, 32)
    k_part, _ = wi.kv_values(3, 0, 1, 20, 10, 2, 32)
    assert torch.equal(k_all[20:30].view(torch.int16), k_part.view(torch.int16))
    vals = (k_all.float() * 128 + 255) / 2
    assert torch.all(vals == vals.round()) and vals.min() >= 0 and vals.max() <= 255


@pytest.mark.parametrize("hd", [32, 64, 128])
def test_page_layout_is_a_bijection(hd):
    for f in (wi.k_page_index, wi.v_page_index):
        idx = f(hd).reshape(-1)
        assert np.array_equal(np.sort(idx), np.arange(16 * hd))
    x = np.random.default_rng(0).standard_normal((3, 16, hd)).astype(np.float32)
    for which in ("k", "v"):
        assert np.array_equal(wi.slots_from_pages(wi.pages_from_slots(x, which), which, hd), x)


def test_workload_mixes():
    m = wi.make_mix("tiny")
    assert m.B == 4 and m.ctx_len.min() >= 32 and m.ctx_len.max() <= 128 and set(m.gamma) <= {1, 2, 3, 4}
    m = wi.make_mix("8b_b32")
    assert m.B == 32 and m.ctx_len.min() >= 512 and m.ctx_len.max() <= 2048
    assert m.gamma.min() >= 1 and m.gamma.max() <= 8 and np.all((m.t_draft >= 0.8) & (m.t_draft <= 1.2))
    m = wi.make_mix("8b_b256")
    assert m.B == 256 and m.ctx_len.min() >= 1024 and m.ctx_len.max() <= 8192 and set(m.gamma) <= set(range(2, 7))
    m = wi.make_mix("8b_dyn128")
    assert m.B == 128 and m.gamma.max() <= 16 and 0.1 < (m.gamma == 0).mean() < 0.4
    assert m.ctx_len.min() >= 256 and m.ctx_len.max() <= 32768 and m.sigma.min() >= 0.2 and m.sigma.max() <= 2
    m = wi.make_mix("70b_b64")
    assert m.B == 64 and m.shape.n_layers == 80 and m.ctx_len.min() >= 1024
    pt, nb = wi.page_table(wi.make_mix("8b_b32"))
    used = pt[pt >= 0]
    assert len(np.unique(used)) == len(used) and used.max() < nb


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_context_kv_placement_agrees_slot_by_slot(dtype):
    """The oracle's host placement (slot-major pages) and the device-side fill (the
    library's page order) put every context position's K and V at the slot the page table
    and the respective layout name (checked one slot at a time), and touch nothing else."""
    import torch
    from oracle import fixtures as fx
    shape = wi.ModelShape("place", 2, 256, 4, 2, 64, 512, 1024, dtype, 1e4)
    mix = wi.custom_mix(shape, [37, 16, 0, 50, 1], [1, 2, 0, 3, 16])
    pt, nb = wi.page_table(mix)
    host = fx.empty_pools(shape, nb)
    fx.place_synthetic_kv(mix, host, pt)
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    dev_k = torch.zeros(shape.n_layers, nb, shape.n_kv_heads, 16 * shape.head_dim, dtype=tdt)
    dev_v = torch.zeros_like(dev_k)
    wi.fill_kv_pool(dev_k, dev_v, mix, pt)
    hd = shape.head_dim
    ref = fx.empty_pools(shape, nb)          # slot-major
    ref_dev = fx.empty_pools(shape, nb)      # the library's page order
    kidx, vidx = wi.k_page_index(hd), wi.v_page_index(hd)
    for i in range(mix.B):
        n = int(mix.ctx_len[i])
        for l in range(shape.n_layers):
            K, V = wi.kv_values(mix.seed, l, i, 0, n, shape.n_kv_heads, hd, "cpu", tdt)
            K, V = fx._to_storage(K, shape), fx._to_storage(V, shape)
            for t in range(n):
                for h in range(shape.n_kv_heads):
                    b, sl = pt[i, t // 16], t % 16
                    ref[0][l, b, h, sl * hd:(sl + 1) * hd] = K[t, h]
                    ref[1][l, b, h, sl * hd:(sl + 1) * hd] = V[t, h]
                    ref_dev[0][l, b, h, kidx[sl]] = K[t, h]
                    ref_dev[1][l, b, h, vidx[sl]] = V[t, h]
    for w, dev in ((0, dev_k), (1, dev_v)):
        np.testing.assert_array_equal(host[w], ref[w])
        np.testing.assert_array_equal(fx._to_storage(dev, shape), ref_dev[w])
