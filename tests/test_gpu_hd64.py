"""bf16 prefill and decode with 64-dimensional heads (the boundary's other
head_dim value) against the float64 oracle: rowwise relative error <= 2e-2 per
token; batch invariance and the shared-prefix layout bit for bit.

Shapes: d = 1024 (16 heads) and d = 1280 (20 heads), two layers.  The small
batches run every GEMM as half tiles; the 8 x 640-row batch (T = 5,120) runs
the QKV and gate/up GEMMs in the ping-pong kernel on whole tiles, so both
epilogues that rotate 64-dimensional heads (a whole tile's eight waves and a
half tile's four) are covered.  d = 1280 is not a multiple of 1,024, so its
decode takes the tile GEMMs instead of the split-K ones."""
import dataclasses

import numpy as np
import pytest

import synth
from oracle import rift_oracle as O
from tests.rift_testlib import (f64, oracle_layer_weights, rowwise_rel_err, shared_layout, torch_mod, upload,
                                upload_layer)

pytestmark = pytest.mark.gpu

TOL = 2e-2


def model(d, ffn, n_layers=2):
    return synth.ModelShape(d=d, n_heads=d // 64, head_dim=64, ffn=ffn, n_layers=n_layers)


@pytest.fixture(scope="module")
def R():
    import paper_2609_29029_amd as R
    torch = torch_mod()
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    R.load()
    return R


def layers_for(m, seed_cid):
    wl = dataclasses.replace(synth.get("one_tile"), model=m, cid=seed_cid)
    return [synth.make_layer(wl, l) for l in range(m.n_layers)]


def cfg_for(R, m):
    return R.model_cfg(m.d, m.n_heads, m.head_dim, m.ffn, m.n_layers, m.rms_eps, m.rope_base, R.RIFT_BF16)


def run_prefill(R, m, Wd, x, cu, pos, n_prefix=0):
    """hidden [T][d] (float64) and the key/value cache [layers][2][T][d] (float32)."""
    torch = torch_mod()
    cfg = cfg_for(R, m)
    T = x.shape[0]
    L = int(np.diff(cu).max()) + (n_prefix if n_prefix else 0)
    ws = torch.empty(R.rift_prefill_workspace_size(cfg, T, L), dtype=torch.uint8, device="cuda")
    kv = torch.empty(m.n_layers, 2, T, m.d, dtype=torch.bfloat16, device="cuda")
    hid = torch.empty(T, m.d, dtype=torch.float32, device="cuda")
    R.rift_prefill(cfg, Wd, upload(x, "bf16"), torch.from_numpy(np.asarray(cu, dtype=np.int32)).cuda(),
                   torch.from_numpy(np.asarray(pos, dtype=np.int32)).cuda(), len(cu) - 1, L, hid, ws,
                   kv_cache=kv, n_prefix=n_prefix)
    torch.cuda.synchronize()
    return hid.cpu().numpy().astype(np.float64), kv.float().cpu().numpy()


@pytest.mark.parametrize("d,ffn,lens,n_check", [(1024, 2816, [7, 130, 300], 3), (1024, 2816, [640] * 8, 2),
                                                 (1280, 3456, [7, 130, 300], 3)])
def test_hd64_prefill_parity_and_batch_invariance(R, d, ffn, lens, n_check):
    """16 heads: attention from the query-block work list; 20 heads (not a
    multiple of 8): one workgroup per (sequence, head) looping over its
    blocks."""
    m = model(d, ffn)
    rng = np.random.default_rng(sum(lens))
    Ws = layers_for(m, 40)
    Wd = [upload_layer(W, "bf16") for W in Ws]
    x = synth.store(rng.standard_normal((sum(lens), m.d)).astype(np.float32), "bf16")
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    pos = np.concatenate([np.arange(l) for l in lens]).astype(np.int32)
    hid, _ = run_prefill(R, m, Wd, x, cu, pos)
    seqs = sorted({0, len(lens) - 1, int(np.argmin(lens))})[:n_check]
    ys = O.prefill(f64(x, "bf16"), cu, pos, [oracle_layer_weights(W, "bf16") for W in Ws], m.n_heads,
                   m.head_dim, m.rms_eps, m.rope_base, seqs)
    for i in seqs:
        err = rowwise_rel_err(hid[cu[i]:cu[i + 1]], ys[i])
        print(f"lens {lens[:3]}...: sequence {i} rowwise rel err {err:.3e}")
        assert err <= TOL, (i, err)
    # the last sequence prefilled alone: the same bits
    i = len(lens) - 1
    alone, _ = run_prefill(R, m, Wd, x[cu[i]:cu[i + 1]], np.array([0, lens[i]]), np.arange(lens[i]))
    assert np.array_equal(alone, hid[cu[i]:cu[i + 1]])


def test_hd64_shared_prefix_matches_unshared(R):
    """Prompts [35 system rows | own rows] packed per prompt and as one shared
    prefix: hidden states and key/value rows equal bit for bit."""
    m = model(1024, 2816)
    rng = np.random.default_rng(64)
    Ws = layers_for(m, 41)
    Wd = [upload_layer(W, "bf16") for W in Ws]
    n_sys, own = 35, [1, 60, 200, 129]
    sysr = synth.store(rng.standard_normal((n_sys, m.d)).astype(np.float32), "bf16")
    rows = [np.concatenate([sysr, synth.store(rng.standard_normal((k, m.d)).astype(np.float32), "bf16")])
            for k in own]
    xa = np.concatenate(rows)
    lens = [n_sys + k for k in own]
    cua = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    posa = np.concatenate([np.arange(l) for l in lens]).astype(np.int32)
    xb, cub, posb = shared_layout(xa, cua, posa, n_sys)
    ha, ka = run_prefill(R, m, Wd, xa, cua, posa)
    hb, kb = run_prefill(R, m, Wd, xb, cub, posb, n_prefix=n_sys)
    for i in range(len(own)):
        a0, a1 = int(cua[i]), int(cua[i + 1])
        b0, b1 = int(cub[i + 1]), int(cub[i + 2])
        assert np.array_equal(ha[a0:a0 + n_sys], hb[:n_sys]), i
        assert np.array_equal(ha[a0 + n_sys:a1], hb[b0:b1]), i
        assert np.array_equal(ka[:, :, a0:a0 + n_sys], kb[:, :, :n_sys]), i
        assert np.array_equal(ka[:, :, a0 + n_sys:a1], kb[:, :, b0:b1]), i


@pytest.mark.parametrize("d,ffn", [(1024, 2816), (1280, 3456)])
def test_hd64_decode_matches_oracle(R, d, ffn):
    """Prefill three prompts with the key/value cache, then three decode steps;
    every generated token's output against the float64 stack run on the
    extended prompt."""
    torch = torch_mod()
    m = model(d, ffn)
    lens, steps = [5, 17, 40], 3
    rng = np.random.default_rng(d)
    Ws = layers_for(m, 42)
    Wd = [upload_layer(W, "bf16") for W in Ws]
    T = sum(lens)
    store = lambda a: synth.store(a.astype(np.float32), "bf16")
    packed = store(rng.standard_normal((T, m.d)))
    new = store(rng.standard_normal((steps, len(lens), m.d)))
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    pos = np.concatenate([np.arange(L) for L in lens]).astype(np.int32)
    cfg = cfg_for(R, m)
    Lmax = max(lens)
    ws = torch.empty(R.rift_prefill_workspace_size(cfg, T, Lmax), dtype=torch.uint8, device="cuda")
    kv = torch.empty(m.n_layers, 2, T, m.d, dtype=torch.bfloat16, device="cuda")
    hid = torch.empty(T, m.d, dtype=torch.float32, device="cuda")
    cu_d = torch.from_numpy(cu).cuda()
    R.rift_prefill(cfg, Wd, upload(packed, "bf16"), cu_d, torch.from_numpy(pos).cuda(), len(lens), Lmax, hid, ws,
                   kv_cache=kv)
    kv_new = torch.full((m.n_layers, 2, len(lens), steps, m.d), float("nan"), dtype=torch.bfloat16, device="cuda")
    dws = torch.empty(R.rift_decode_workspace_size(cfg, len(lens), Lmax, steps), dtype=torch.uint8, device="cuda")
    outs = []
    for t in range(steps):
        out = torch.empty(len(lens), m.d, dtype=torch.float32, device="cuda")
        R.rift_decode_step(cfg, Wd, upload(new[t], "bf16"), cu_d, T, Lmax, kv, kv_new, t, out, dws)
        outs.append(out)
    torch.cuda.synchronize()
    Wo = [oracle_layer_weights(W, "bf16") for W in Ws]
    P64, N64 = f64(packed, "bf16"), f64(new, "bf16")
    for i, L in enumerate(lens):
        ref = O.decode_outputs(P64[cu[i]:cu[i + 1]], N64[:, i], Wo, m.n_heads, m.head_dim, m.rms_eps, m.rope_base)
        got = np.stack([o[i].cpu().numpy().astype(np.float64) for o in outs])
        err = rowwise_rel_err(got, ref)
        print(f"d={d} prompt {i} (L={L}): decode rel err {err:.3e}")
        assert err <= TOL, (i, err)


def test_hd64_attention_worklist_many_sequences(R):
    """Eight heads (one group of eight: the query-block work list) over 1,100
    sequences, which the list kernel scans 1,024 at a time, empty ones among
    them: sequences on both sides of the 1,024 boundary and the last against
    the oracle, and one prefilled alone gives the same bits."""
    m = model(512, 1408)
    rng = np.random.default_rng(1100)
    lens = [int(v) for v in rng.integers(1, 41, size=1100)]
    lens[0], lens[5], lens[1023], lens[1024], lens[1030] = 130, 0, 0, 200, 0
    Ws = layers_for(m, 41)
    Wd = [upload_layer(W, "bf16") for W in Ws]
    x = synth.store(rng.standard_normal((sum(lens), m.d)).astype(np.float32), "bf16")
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    pos = np.concatenate([np.arange(l) for l in lens]).astype(np.int32)
    hid, _ = run_prefill(R, m, Wd, x, cu, pos)
    seqs = [0, 1022, 1024, 1099]
    ys = O.prefill(f64(x, "bf16"), cu, pos, [oracle_layer_weights(W, "bf16") for W in Ws], m.n_heads,
                   m.head_dim, m.rms_eps, m.rope_base, seqs)
    for i in seqs:
        err = rowwise_rel_err(hid[cu[i]:cu[i + 1]], ys[i])
        print(f"sequence {i} (L={lens[i]}): rowwise rel err {err:.3e}")
        assert err <= TOL, (i, err)
    i = 1024
    alone, _ = run_prefill(R, m, Wd, x[cu[i]:cu[i + 1]], np.array([0, lens[i]]), np.arange(lens[i]))
    assert np.array_equal(alone, hid[cu[i]:cu[i + 1]])
