"""GPU parity of the compaction, soft-embedding and unmasking kernels
against the oracle (bit-exact for integer work)."""
import itertools

import numpy as np
import pytest
import torch

from oracle import selection as S
from oracle import embed as E
from oracle import unmask as U
from synthetic import WORKLOADS, seeded_normal, seeded_uniform_ints

pytestmark = pytest.mark.gpu


def _select_gpu(P0, G, b, j, Lb, Mb, mode, Tb, incl, tokens, tmode=0):
    from paper_2608_23167_amd.api import select_params, ssm_select_suffix
    B = tokens.shape[0]
    cap = P0 + G + 8
    pos = torch.full((cap,), -7, dtype=torch.int32, device="cuda")
    tok_c = torch.full((B, cap), -7, dtype=torch.int32, device="cuda")
    region = torch.full((cap,), -7, dtype=torch.int8, device="cuda")
    n, ns, f = ssm_select_suffix(select_params(P0, G, b, j, Lb, Mb, mode, Tb, incl, tmode), tokens,
                                 pos, tok_c, region)
    torch.cuda.synchronize()
    return n, ns, f, pos.cpu().numpy(), region.cpu().numpy(), tok_c.cpu().numpy()


@pytest.mark.parametrize("name", list(WORKLOADS))
def test_select_matches_oracle_on_workloads(gpu, name):
    wl = WORKLOADS[name]
    B = min(wl.batch, 2)
    tokens = seeded_uniform_ints((B, wl.total_len), 0, wl.model.vocab, 1, "sel").to("cuda")
    tok_np = tokens.cpu().numpy()
    for j in range(wl.n_blocks):
        for incl in (True, False):
            c = S.compacted_rows(wl.prompt_len, wl.gen_len, wl.block_size, j, wl.local_budget,
                                 wl.middle_budget, wl.middle_mode, wl.tail_budget, incl)
            n, ns, f, pos, reg, tc = _select_gpu(wl.prompt_len, wl.gen_len, wl.block_size, j,
                                                 wl.local_budget, wl.middle_budget,
                                                 wl.middle_mode, wl.tail_budget, incl, tokens)
            assert (n, ns, f) == (len(c.pos), c.n_suffix, c.first_out_row)
            assert np.array_equal(pos[:n], c.pos)
            assert np.array_equal(reg[:n], c.region)
            assert np.all(pos[n:] == -7)   # nothing written past the rows
            for s in range(B):
                assert np.array_equal(tc[s, :n], tok_np[s, c.pos])


def test_select_brute_force_sweep(gpu):
    """Every middle mode (strided, block start, block end, both) and tail mode
    (spread, start only), local budgets that cut a block included."""
    tokens = seeded_uniform_ints((1, 5 + 64), 0, 1000, 2, "sweep").to("cuda")
    tok_np = tokens.cpu().numpy()
    cases = 0
    for b, nb in ((4, 16), (8, 8), (1, 12), (3, 7)):
        G = b * nb
        for j in range(nb):
            for Lb, mode, Tb, tmode in itertools.product((0, 1, b, b + 2, 3 * b + 1, G), range(4),
                                                         (0, 1, 2, 3, b), (0, 1)):
                for Mb in ((0, 2, 5, G) if mode == S.MIDDLE_STRIDED else (0,)):
                    c = S.compacted_rows(5, G, b, j, Lb, Mb, mode, Tb, True, tmode)
                    n, ns, f, pos, reg, tc = _select_gpu(5, G, b, j, Lb, Mb, mode, Tb, True,
                                                         tokens[:, :5 + G].contiguous(), tmode)
                    assert n == len(c.pos) and ns == c.n_suffix
                    assert np.array_equal(pos[:n], c.pos), (b, j, Lb, Mb, Tb, mode, tmode)
                    assert np.array_equal(reg[:n], c.region)
                    assert np.array_equal(tc[0, :n], tok_np[0, c.pos])
                    cases += 1
    print(f"[select sweep] {cases} cases", flush=True)


@pytest.mark.parametrize("dtype,d,V,k", [("f32", 128, 512, 5), ("bf16", 4096, 2048, 5),
                                         ("bf16", 3584, 1024, 8), ("f32", 64, 100, 1)])
def test_embed_matches_oracle(gpu, dtype, d, V, k):
    from paper_2608_23167_amd.api import ssm_embed_suffix
    from paper_2608_23167_amd.model import DeviceModel
    from synthetic.configs import ModelShape
    from synthetic.generate import ModelWeights
    tdt = torch.float32 if dtype == "f32" else torch.bfloat16
    shape = ModelShape("emb", 0, d, 1, 1, d, 1, V, V - 1, dtype=dtype)
    Emb = seeded_normal((V, d), 3, "emb", 0.02, dtype=tdt)
    mw = ModelWeights(shape, Emb.cuda(), torch.ones(d, dtype=tdt, device="cuda"), Emb.cuda(), [])
    dm = DeviceModel(shape, mw)
    B, Lt = 2, 96
    P0, G, b, j = 16, 80, 16, 0
    c = S.compacted_rows(P0, G, b, j, 16, 6, 0, 4, True)
    n = len(c.pos)
    rng = np.random.default_rng(5)
    tokens = rng.integers(0, V - 1, size=(B, Lt)).astype(np.int32)
    tokens[:, P0:] = V - 1
    tokens[:, P0 + 3] = 7   # a decoded token inside the block
    pred_ids = rng.integers(0, V, size=(B, Lt, k)).astype(np.int32)
    w = rng.random((B, Lt, k)).astype(np.float32)
    pred_w = (w / w.sum(-1, keepdims=True)).astype(np.float32)
    pred_step = rng.choice([2, 3, -1], size=(B, Lt)).astype(np.int32)
    alpha = 0.4
    tok_c = np.stack([tokens[s, c.pos] for s in range(B)]).astype(np.int32)
    x = torch.zeros(B * n * d, dtype=torch.float32, device="cuda")
    ssm_embed_suffix(dm, torch.from_numpy(tok_c).cuda(), torch.from_numpy(c.pos).cuda(),
                     torch.from_numpy(c.region).cuda(), n, torch.from_numpy(pred_ids).cuda(),
                     torch.from_numpy(pred_w).cuda(), torch.from_numpy(pred_step).cuda(), 3, k,
                     alpha, x)
    got = x.view(B, n, d).cpu().numpy()
    En = Emb.double().numpy()
    for s in range(B):
        ref = E.embed_rows(En, tokens[s], c.pos, c.region, pred_ids[s], pred_w[s].astype(np.float64),
                           pred_step[s], 3, alpha, V - 1)
        assert np.max(np.abs(got[s] - ref)) < 1e-6
        soft_rows = (c.region >= S.REGION_LOCAL) & (pred_step[s][c.pos] == 3)
        assert soft_rows.any()
        # rows without a prediction are bit-exact table rows
        for r in np.nonzero(~soft_rows)[0]:
            assert np.array_equal(got[s, r], Emb[tok_c[s, r]].float().numpy())


@pytest.mark.parametrize("rule", ["topn", "threshold", "margin"])
def test_unmask_matches_oracle(gpu, rule):
    from paper_2608_23167_amd.api import ssm_unmask
    from paper_2608_23167_amd.decoder import RULES
    rng = np.random.default_rng({"topn": 1, "threshold": 2, "margin": 3}[rule])
    B, b, k, Lt, mask = 3, 32, 4, 200, 999
    for trial in range(20):
        P = 64
        n_suf = int(rng.integers(0, 40))
        n_out = b + n_suf
        tokens = rng.integers(0, 900, size=(B, Lt)).astype(np.int32)
        tokens[:, P:] = mask
        done = rng.random((B, b)) < 0.4
        tokens[:, P:P + b][done] = 5
        conf = rng.random((B, n_out)).astype(np.float32)
        if trial % 3 == 0:
            conf[:, : b // 2] = 0.95   # ties
        w = np.sort(rng.random((B, n_out, k)), axis=-1)[..., ::-1].astype(np.float32)
        w = w / w.sum(-1, keepdims=True)
        argmax = rng.integers(0, 900, size=(B, n_out)).astype(np.int32)
        topk_ids = rng.integers(0, 900, size=(B, n_out, k)).astype(np.int32)
        pos_out = np.concatenate([np.arange(P, P + b), np.sort(rng.choice(np.arange(P + b, Lt), n_suf, replace=False))]).astype(np.int32)
        n_per = int(rng.integers(1, 9))
        thr = float(rng.choice([0.5, 0.9, 0.99, 0.0]))
        t_dev = torch.from_numpy(tokens).cuda()
        pred_ids = torch.zeros((B, Lt, k), dtype=torch.int32, device="cuda")
        pred_w = torch.zeros((B, Lt, k), dtype=torch.float32, device="cuda")
        pred_step = torch.full((B, Lt), -1, dtype=torch.int32, device="cuda")
        sel = torch.zeros(B * b, dtype=torch.uint8, device="cuda")
        left = torch.zeros(B, dtype=torch.int32, device="cuda")
        ssm_unmask(t_dev, P, b, mask, RULES[rule], n_per, thr, torch.from_numpy(argmax).cuda(),
                   torch.from_numpy(conf).cuda(), torch.from_numpy(topk_ids).cuda(),
                   torch.from_numpy(w).cuda(), k, n_out, torch.from_numpy(pos_out).cuda(), 11,
                   pred_ids, pred_w, pred_step, sel, left)
        got = t_dev.cpu().numpy()
        for s in range(B):
            masked = tokens[s, P:P + b] == mask
            # the kernel's margin in float32, as the decision is taken in that precision
            margin = (conf[s, :b] * (np.float32(1) - w[s, :b, 1] / w[s, :b, 0])).astype(np.float32)
            want = U.choose(conf[s, :b], masked, rule, n_per, thr, margin)
            assert np.array_equal(sel.view(B, b)[s].cpu().numpy().astype(bool), want)
            exp_tok = tokens[s].copy()
            exp_tok[P:P + b][want] = argmax[s, :b][want]
            assert np.array_equal(got[s], exp_tok)
            assert left[s].item() == int(masked.sum() - want.sum())
            ps = pred_step[s].cpu().numpy()
            assert np.all(ps[pos_out[b:]] == 11)
            others = np.setdiff1d(np.arange(Lt), pos_out[b:])
            assert np.all(ps[others] == -1)
            assert np.array_equal(pred_ids[s].cpu().numpy()[pos_out[b:]], topk_ids[s, b:])
            assert np.array_equal(pred_w[s].cpu().numpy()[pos_out[b:]], w[s, b:])


def test_early_stop_matches_oracle(gpu):
    """Early termination kernel: bit-exact fill and done flags against the
    oracle, over sequences with and without the end id, some already done,
    for every block of the sequence."""
    from oracle import generate as OG
    from paper_2608_23167_amd.api import ssm_early_stop
    B, L, b, eos, P0 = 6, 5 + 8 * 16, 16, 11, 5
    for seed in range(3):
        tok = seeded_uniform_ints((B, L), 0, 40, 10 + seed, "es").numpy()
        tok[tok == eos] = eos + 1
        rng = np.random.default_rng(seed)
        for s in range(B):                       # plant the end id in some blocks
            for _ in range(rng.integers(0, 3)):
                tok[s, rng.integers(P0, L)] = eos
        done = (rng.random(B) < 0.2)
        t_dev = torch.from_numpy(tok).to("cuda")
        d_dev = torch.from_numpy(done.astype(np.int32)).to("cuda")
        for j in range(8):
            start = P0 + j * b
            all_done = OG.early_stop(tok, done, start, b, eos)
            ssm_early_stop(t_dev, start, b, eos, d_dev)
            torch.cuda.synchronize()
            assert np.array_equal(t_dev.cpu().numpy(), tok), (seed, j)
            assert np.array_equal(d_dev.cpu().numpy().astype(bool), done), (seed, j)
            assert all_done == bool(done.all())
