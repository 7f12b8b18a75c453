"""GPU checks of repacking on one GPU: the page migration kernel bit for bit
against the oracle's copy, and a whole repack (plan, page assignment,
migration) after which every moved trajectory's attention is unchanged."""
import numpy as np
import pytest
import torch

from oracle import decode_attention_from_host
from oracle.repack import best_fit_consolidation, migrate_pages
from workloads import custom_config, host_arrays, make_workload

pytestmark = pytest.mark.gpu


def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("needs a GPU")


def _say(msg):
    print(f"[gpu-repack] {msg}", flush=True)


def host(t):
    t = t.detach().cpu()
    if t.dtype == torch.bfloat16:
        return t.view(torch.int16).numpy().view(np.uint16)
    return t.numpy()


@pytest.mark.parametrize("page_bytes", [4, 12, 16, 48, 4096, 16384, 65536 + 16])
def test_migrate_pages_bit_exact(page_bytes):
    from paper_2510_12633_amd import _native as N
    _need_gpu()
    _say(f"migrate page_bytes={page_bytes}")
    rng = np.random.default_rng(page_bytes)
    n_src, n_dst = 300, 500
    src = torch.randint(0, 256, (n_src, page_bytes), dtype=torch.uint8,
                        device="cuda")
    dst = torch.randint(0, 256, (n_dst, page_bytes), dtype=torch.uint8,
                        device="cuda")
    k = 200
    pairs = np.stack([rng.integers(0, n_src, k),
                      rng.permutation(n_dst)[:k]], axis=1).astype(np.int32)
    pairs[5] = [-1, pairs[5, 1]]                    # skipped: source out of range
    pairs[9] = [pairs[9, 0], n_dst + 3]             # skipped: destination out of range
    want = migrate_pages(host(src), host(dst),
                         pairs[(pairs[:, 0] >= 0) & (pairs[:, 1] < n_dst)])
    N.laminar_migrate_pages(src, n_src, dst, n_dst, page_bytes,
                            torch.as_tensor(pairs, device="cuda"), k,
                            torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert np.array_equal(host(dst), want)


def _rollouts(kv_dtype, seed):
    """Six rollouts (own pools of 160 pages) in their ramp-down phase."""
    rng = np.random.default_rng(seed)
    rolls = []
    for r in range(6):
        n = int(rng.integers(1, 4))
        lens = [int(x) for x in rng.integers(1, 600, n)]
        cfg = custom_config(lens, 28, 4, 128, kv_dtype=kv_dtype, pool_pages=160)
        rolls.append(make_workload(cfg, seed=100 + r, device="cuda"))
    return rolls


@pytest.mark.parametrize("kv_dtype", ["bf16", "fp8_e4m3fn"])
def test_repack_moves_trajectories_without_changing_attention(kv_dtype):
    from paper_2510_12633_amd import _native as N
    from paper_2510_12633_amd.api import PagedDecodeAttention, migrate
    _need_gpu()
    rolls = _rollouts(kv_dtype, seed=3 if kv_dtype == "bf16" else 4)

    def attend(wl, q, table, lens, pools):
        kp, vp, ks, vs = pools
        att = PagedDecodeAttention(
            batch=len(lens), num_q_heads=28, num_kv_heads=4, head_dim=128,
            num_pages=kp.shape[0], max_blocks_per_seq=table.shape[1],
            seq_lens_host=lens, softmax_scale=wl.softmax_scale,
            kv_dtype=kv_dtype, k_scale=ks, v_scale=vs)
        out, lse = att(q, kp, vp, torch.as_tensor(table, device="cuda"),
                       torch.as_tensor(lens, device="cuda"))
        torch.cuda.synchronize()
        res = out.cpu().numpy(), lse.cpu().numpy()
        att.close()
        return res

    before = [attend(w, w.q, w.block_table, w.seq_lens,
                     (w.k_pages, w.v_pages, w.k_scale, w.v_scale)) for w in rolls]
    used = [int(np.unique(w.block_table[w.block_table >= 0]).size) for w in rolls]
    prev = [u + 5 for u in used]
    reqs = [w.batch for w in rolls]
    plan = N.laminar_repack_plan(used, prev, reqs, 160, 12)
    assert plan == best_fit_consolidation(used, prev, reqs, 160, 12)
    assert plan, "the scenario should move something"
    _say(f"{kv_dtype}: plan {plan} (usage {used})")

    # destination state: its own trajectories, then the moved ones
    state = {d: dict(q=[rolls[d].q], table=[rolls[d].block_table],
                     lens=[rolls[d].seq_lens], who=[(d, i) for i in range(rolls[d].batch)],
                     taken=set(np.unique(rolls[d].block_table[rolls[d].block_table >= 0]).tolist()))
             for _, d in plan}
    for s, d in plan:
        src, dst, st = rolls[s], rolls[d], state[d]
        free = np.array([p for p in range(dst.num_pages) if p not in st["taken"]],
                        np.int32)
        width = max(max(t.shape[1] for t in st["table"]), src.block_table.shape[1])
        table, pairs, n_used = N.laminar_migration_pairs(
            src.block_table, src.seq_lens, free, width)
        st["taken"].update(free[:n_used].tolist())
        host_before = [host(x) for x in (dst.k_pages, dst.v_pages)]
        migrate((src.k_pages, src.v_pages, src.k_scale, src.v_scale),
                (dst.k_pages, dst.v_pages, dst.k_scale, dst.v_scale),
                torch.as_tensor(pairs, device="cuda"))
        torch.cuda.synchronize()
        for got, pool_src, pool_dst in zip((dst.k_pages, dst.v_pages),
                                           (src.k_pages, src.v_pages), host_before):
            assert np.array_equal(host(got),
                                  migrate_pages(host(pool_src), pool_dst, pairs))
        st["q"].append(src.q)
        st["table"].append(table)
        st["lens"].append(src.seq_lens)
        st["who"] += [(s, i) for i in range(src.batch)]

    for d, st in state.items():
        width = max(t.shape[1] for t in st["table"])
        table = np.concatenate([np.pad(t, ((0, 0), (0, width - t.shape[1])),
                                       constant_values=-1) for t in st["table"]])
        lens = np.concatenate(st["lens"]).astype(np.int32)
        q = torch.cat(st["q"])
        dw = rolls[d]
        out, lse = attend(dw, q, table, lens,
                          (dw.k_pages, dw.v_pages, dw.k_scale, dw.v_scale))
        for row, (r, i) in enumerate(st["who"]):
            eo = np.abs(out[row] - before[r][0][i]).max()
            el = np.abs(lse[row] - before[r][1][i]).max()
            assert eo <= 1e-5 and el <= 1e-5, (d, r, i, eo, el)
        arrays = dict(host_arrays(dw), q=host(q), block_table=table, seq_lens=lens)
        ro, rl = decode_attention_from_host(arrays)
        assert np.abs(out - ro).max() <= 1e-3 and np.abs(lse - rl).max() <= 1e-3
        _say(f"{kv_dtype}: destination {d} holds {len(st['who'])} trajectories, "
             f"attention unchanged")
