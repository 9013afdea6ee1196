"""Decode after prefill (reading R15) against the oracle: three prompts of
LLaMA-7B width, two layers, prefill with the key/value cache, then three
decode steps; every generated token's output within the bf16 gate (2e-2,
rowwise) of the float64 decoder stack run on the extended prompt."""
import dataclasses

import numpy as np
import pytest

import synth
from oracle import rift_oracle as O
from tests.rift_testlib import f64, oracle_layer_weights, rowwise_rel_err, torch_mod, upload, upload_layer

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def R():
    import paper_2609_29029_amd as R
    torch = torch_mod()
    assert torch.cuda.is_available(), "GPU tests need a GPU"
    R.load()
    return R


def test_decode_steps_match_the_extended_prefill(R):
    torch = torch_mod()
    w = synth.get("one_tile")
    m = w.model
    n_layers, lens, steps = 2, [5, 17, 40], 3
    rng = np.random.default_rng(0x52494654)
    T = sum(lens)
    store = lambda a: synth.store(a.astype(np.float32), "bf16")
    packed = store(rng.standard_normal((T, m.d)))
    new = store(rng.standard_normal((steps, len(lens), m.d)))
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    pos = np.concatenate([np.arange(L) for L in lens]).astype(np.int32)
    Ws = [synth.make_layer(w, l) for l in range(n_layers)]
    Wd = [upload_layer(W, "bf16") for W in Ws]
    cfg = R.model_cfg(m.d, m.n_heads, m.head_dim, m.ffn, n_layers, m.rms_eps, m.rope_base, R.RIFT_BF16)
    Lmax = max(lens)
    ws = torch.empty(R.rift_prefill_workspace_size(cfg, T, Lmax), dtype=torch.uint8, device="cuda")
    kv = torch.empty(n_layers, 2, T, m.d, dtype=torch.bfloat16, device="cuda")
    hid = torch.empty(T, m.d, dtype=torch.float32, device="cuda")
    cu_d = torch.from_numpy(cu).cuda()
    R.rift_prefill(cfg, Wd, upload(packed, "bf16"), cu_d, torch.from_numpy(pos).cuda(), len(lens), Lmax, hid, ws,
                   kv_cache=kv)
    kv_new = torch.full((n_layers, 2, len(lens), steps, m.d), float("nan"), dtype=torch.bfloat16, device="cuda")
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
        print(f"prompt {i} (L={L}): decode rel err {err:.3e}")
        assert err <= 2e-2, (i, err)


def test_decode_is_batch_invariant(R):
    """A prompt's decode output does not depend on the other prompts of the
    call (prefill and decode), bit for bit."""
    torch = torch_mod()
    w = synth.get("one_tile")
    m = w.model
    rng = np.random.default_rng(5)
    store = lambda a: synth.store(a.astype(np.float32), "bf16")
    lens = [9, 30]
    T = sum(lens)
    packed = store(rng.standard_normal((T, m.d)))
    x_next = store(rng.standard_normal((2, m.d)))
    W = upload_layer(synth.make_layer(w, 0), "bf16")
    cfg = R.model_cfg(m.d, m.n_heads, m.head_dim, m.ffn, 1, m.rms_eps, m.rope_base, R.RIFT_BF16)

    def run(sel):
        ls = [lens[i] for i in sel]
        rows = np.concatenate([packed[sum(lens[:i]):sum(lens[:i + 1])] for i in sel])
        cu = torch.tensor(np.concatenate([[0], np.cumsum(ls)]), dtype=torch.int32, device="cuda")
        pos = torch.tensor(np.concatenate([np.arange(L) for L in ls]), dtype=torch.int32, device="cuda")
        Tn = int(sum(ls))
        ws = torch.empty(R.rift_prefill_workspace_size(cfg, Tn, max(ls)), dtype=torch.uint8, device="cuda")
        kv = torch.empty(1, 2, Tn, m.d, dtype=torch.bfloat16, device="cuda")
        hid = torch.empty(Tn, m.d, dtype=torch.float32, device="cuda")
        R.rift_prefill(cfg, [W], upload(rows, "bf16"), cu, pos, len(ls), max(ls), hid, ws, kv_cache=kv)
        kvn = torch.empty(1, 2, len(ls), 1, m.d, dtype=torch.bfloat16, device="cuda")
        dws = torch.empty(R.rift_decode_workspace_size(cfg, len(ls), max(ls), 1), dtype=torch.uint8, device="cuda")
        out = torch.empty(len(ls), m.d, dtype=torch.float32, device="cuda")
        R.rift_decode_step(cfg, [W], upload(x_next[list(sel)], "bf16"), cu, Tn, max(ls), kv, kvn, 0, out, dws)
        torch.cuda.synchronize()
        return out.cpu().numpy()

    both = run([0, 1])
    alone = run([1])
    assert np.array_equal(both[1], alone[0])


def _decode_case(R, m, lens, steps, n_layers, seed):
    """Prefill `lens` prompts, then `steps` decode steps; returns the inputs
    and the decode outputs [steps][n_seq][d]."""
    torch = torch_mod()
    rng = np.random.default_rng(seed)
    store = lambda a: synth.store(a.astype(np.float32), "bf16")
    T = sum(lens)
    packed = store(rng.standard_normal((T, m.d)))
    new = store(rng.standard_normal((steps, len(lens), m.d)))
    cu = np.concatenate([[0], np.cumsum(lens)]).astype(np.int32)
    pos = np.concatenate([np.arange(L) for L in lens]).astype(np.int32)
    wl = dataclasses.replace(synth.get("one_tile"), model=m)
    Ws = [synth.make_layer(wl, l) for l in range(n_layers)]
    Wd = [upload_layer(W, "bf16") for W in Ws]
    cfg = R.model_cfg(m.d, m.n_heads, m.head_dim, m.ffn, n_layers, m.rms_eps, m.rope_base, R.RIFT_BF16)
    Lmax = max(lens)
    ws = torch.empty(R.rift_prefill_workspace_size(cfg, T, Lmax), dtype=torch.uint8, device="cuda")
    kv = torch.empty(n_layers, 2, T, m.d, dtype=torch.bfloat16, device="cuda")
    hid = torch.empty(T, m.d, dtype=torch.float32, device="cuda")
    cu_d = torch.from_numpy(cu).cuda()
    R.rift_prefill(cfg, Wd, upload(packed, "bf16"), cu_d, torch.from_numpy(pos).cuda(), len(lens), Lmax, hid, ws,
                   kv_cache=kv)
    kv_new = torch.full((n_layers, 2, len(lens), steps, m.d), float("nan"), dtype=torch.bfloat16, device="cuda")
    dws = torch.empty(R.rift_decode_workspace_size(cfg, len(lens), Lmax, steps), dtype=torch.uint8, device="cuda")
    outs = []
    for t in range(steps):
        out = torch.empty(len(lens), m.d, dtype=torch.float32, device="cuda")
        R.rift_decode_step(cfg, Wd, upload(new[t], "bf16"), cu_d, T, Lmax, kv, kv_new, t, out, dws)
        outs.append(out)
    torch.cuda.synchronize()
    got = np.stack([o.cpu().numpy().astype(np.float64) for o in outs])
    return packed, new, cu, Ws, got


def test_decode_narrow_model_tile_path(R):
    """d = 1280 (not a multiple of 1024): the decode GEMMs take the prefill's
    tile kernels instead of the split-K ones; same oracle bar."""
    m = synth.ModelShape(d=1280, n_heads=10, head_dim=128, ffn=3456, n_layers=2)
    lens, steps = [3, 21], 2
    packed, new, cu, Ws, got = _decode_case(R, m, lens, steps, 2, 11)
    Wo = [oracle_layer_weights(W, "bf16") for W in Ws]
    P64, N64 = f64(packed, "bf16"), f64(new, "bf16")
    for i in range(len(lens)):
        ref = O.decode_outputs(P64[cu[i]:cu[i + 1]], N64[:, i], Wo, m.n_heads, m.head_dim, m.rms_eps, m.rope_base)
        err = rowwise_rel_err(got[:, i], ref)
        print(f"prompt {i}: decode rel err {err:.3e}")
        assert err <= 2e-2, (i, err)


def test_decode_two_row_tiles(R):
    """130 prompts (two 128-row tiles of the split-K GEMMs): sampled prompts
    from both tiles against the oracle, and the last prompt's output the same
    bit for bit when it is decoded alone."""
    torch = torch_mod()
    m = synth.get("one_tile").model
    rng = np.random.default_rng(12)
    lens = [int(x) for x in rng.integers(1, 7, size=130)]
    packed, new, cu, Ws, got = _decode_case(R, m, lens, 1, 1, 13)
    Wo = [oracle_layer_weights(W, "bf16") for W in Ws]
    P64, N64 = f64(packed, "bf16"), f64(new, "bf16")
    for i in (0, 77, 127, 128, 129):
        ref = O.decode_outputs(P64[cu[i]:cu[i + 1]], N64[:, i], Wo, m.n_heads, m.head_dim, m.rms_eps, m.rope_base)
        err = rowwise_rel_err(got[:, i], ref)
        print(f"prompt {i} (L={lens[i]}): decode rel err {err:.3e}")
        assert err <= 2e-2, (i, err)
    # prompt 129 alone: same weights, same rows
    W = upload_layer(Ws[0], "bf16")
    cfg = R.model_cfg(m.d, m.n_heads, m.head_dim, m.ffn, 1, m.rms_eps, m.rope_base, R.RIFT_BF16)
    L = lens[129]
    rows = packed[cu[129]:cu[130]]
    ws = torch.empty(R.rift_prefill_workspace_size(cfg, L, L), dtype=torch.uint8, device="cuda")
    kv = torch.empty(1, 2, L, m.d, dtype=torch.bfloat16, device="cuda")
    hid = torch.empty(L, m.d, dtype=torch.float32, device="cuda")
    cu1 = torch.tensor([0, L], dtype=torch.int32, device="cuda")
    R.rift_prefill(cfg, [W], upload(rows, "bf16"), cu1, torch.arange(L, dtype=torch.int32, device="cuda"), 1, L,
                   hid, ws, kv_cache=kv)
    kvn = torch.empty(1, 2, 1, 1, m.d, dtype=torch.bfloat16, device="cuda")
    dws = torch.empty(R.rift_decode_workspace_size(cfg, 1, L, 1), dtype=torch.uint8, device="cuda")
    out = torch.empty(1, m.d, dtype=torch.float32, device="cuda")
    R.rift_decode_step(cfg, [W], upload(new[0, 129:130], "bf16"), cu1, L, L, kv, kvn, 0, out, dws)
    torch.cuda.synchronize()
    assert np.array_equal(out.cpu().numpy()[0].astype(np.float64), got[0, 129])


def test_decode_after_shared_prefix_matches_unshared(R):
    """Decode after a prefill whose system rows were shared (n_prefix) gives
    the same outputs, bit for bit, as after the per-prompt packing: the prompt's
    keys are the prefix rows then its own, in the same order."""
    torch = torch_mod()
    w = synth.get("one_tile")
    m = w.model
    rng = np.random.default_rng(21)
    store = lambda a: synth.store(a.astype(np.float32), "bf16")
    P, own = 6, [4, 11, 0, 1]   # a prompt with no rows after the prefix too
    prefix = store(rng.standard_normal((P, m.d)))
    rows = [store(rng.standard_normal((L, m.d))).reshape(L, m.d) for L in own]
    steps = 2
    new = store(rng.standard_normal((steps, len(own), m.d)))
    W = upload_layer(synth.make_layer(w, 0), "bf16")
    cfg = R.model_cfg(m.d, m.n_heads, m.head_dim, m.ffn, 1, m.rms_eps, m.rope_base, R.RIFT_BF16)
    Lmax = P + max(own)

    def run(shared):
        if shared:
            x = np.concatenate([prefix] + rows)
            cu = np.concatenate([[0, P], P + np.cumsum(own)])
            pos = np.concatenate([np.arange(P)] + [P + np.arange(L) for L in own])
            n_seq = len(own) + 1
        else:
            x = np.concatenate([np.concatenate([prefix, r]) for r in rows])
            cu = np.concatenate([[0], np.cumsum([P + L for L in own])])
            pos = np.concatenate([np.arange(P + L) for L in own])
            n_seq = len(own)
        T = x.shape[0]
        cu_d = torch.tensor(cu, dtype=torch.int32, device="cuda")
        ws = torch.empty(R.rift_prefill_workspace_size(cfg, T, Lmax), dtype=torch.uint8, device="cuda")
        kv = torch.empty(1, 2, T, m.d, dtype=torch.bfloat16, device="cuda")
        hid = torch.empty(T, m.d, dtype=torch.float32, device="cuda")
        R.rift_prefill(cfg, [W], upload(x, "bf16"), cu_d, torch.tensor(pos, dtype=torch.int32, device="cuda"),
                       n_seq, Lmax, hid, ws, kv_cache=kv, n_prefix=P if shared else 0)
        kvn = torch.empty(1, 2, len(own), steps, m.d, dtype=torch.bfloat16, device="cuda")
        dws = torch.empty(R.rift_decode_workspace_size(cfg, len(own), Lmax, steps), dtype=torch.uint8,
                          device="cuda")
        outs = []
        for t in range(steps):
            out = torch.empty(len(own), m.d, dtype=torch.float32, device="cuda")
            R.rift_decode_step(cfg, [W], upload(new[t], "bf16"), cu_d, T, Lmax, kv, kvn, t, out, dws,
                               n_prefix=P if shared else 0)
            outs.append(out)
        torch.cuda.synchronize()
        return np.stack([o.cpu().numpy() for o in outs])

    a, b = run(False), run(True)
    assert np.array_equal(a, b)
