"""GPU parity of the uncompressed decode baseline against the oracle's
dense decode (every row; inputs are bf16-exact, accumulation fp32)."""

import numpy as np
import pytest
import torch

from oracle import dense as odense
from workloads.inputs import to_storage

pytestmark = pytest.mark.gpu

TOL = 1e-4      # row inf-norm relative error: fp32 accumulation over bf16-exact inputs


def _case(Hq, Hkv, d, lens, seed, permute=True):
    g = np.random.default_rng(seed)
    pages = [-(-T // 64) for T in lens]
    total = max(1, sum(pages))
    phys = g.permutation(total) if permute else np.arange(total)
    table = np.zeros((len(lens), max(pages + [1])), dtype=np.int32)
    pos = 0
    for b, n in enumerate(pages):
        table[b, :n] = phys[pos:pos + n]
        pos += n
    pool = odense.new_pool(total, Hkv, d, dtype=np.float32)
    for b, T in enumerate(lens):
        K = to_storage(g.standard_normal((T, Hkv, d)), "bf16")
        V = to_storage(g.standard_normal((T, Hkv, d)), "bf16")
        odense.pack(pool, table, b, 0, K, V)
    q = g.standard_normal((len(lens), Hq, d)).astype(np.float32)
    return pool, table, q


CASES = [
    # (H_q, H_kv, d_h, lengths, split)
    (8, 8, 128, [300, 64, 1, 0, 129], 128),     # MHA, ragged, one-token and empty sequences
    (16, 4, 128, [1000, 777], 256),             # GQA, 4 queries a KV head
    (32, 4, 64, [517, 70], 64),                 # GQA, 8 queries a KV head, d_h 64
    (6, 3, 256, [200, 65], 0),                  # d_h 256, automatic split
    (4, 4, 128, [2049], 0),
]


@pytest.mark.parametrize("Hq, Hkv, d, lens, split", CASES)
def test_dense_decode_all_rows(Hq, Hkv, d, lens, split):
    from paper_2607_24331_amd import dense_decode
    pool, table, q = _case(Hq, Hkv, d, lens, seed=Hq + d + len(lens))
    got = dense_decode(torch.from_numpy(q).cuda(), torch.from_numpy(pool).to(torch.bfloat16).cuda(),
                       torch.from_numpy(table).cuda(),
                       torch.tensor(lens, dtype=torch.int32).cuda(), max(lens), Hkv,
                       split_tokens=split)
    torch.cuda.synchronize()
    got = got.cpu().numpy().astype(np.float64)
    ref = odense.decode(q.astype(np.float64), pool.astype(np.float64), table, lens, Hkv)
    errs = []
    for b, T in enumerate(lens):
        for h in range(Hq):
            if T == 0:
                assert np.all(got[b, h] == 0)
                continue
            errs.append(np.max(np.abs(got[b, h] - ref[b, h])) / np.max(np.abs(ref[b, h])))
    print(f"[dense] H {Hq}/{Hkv} d {d} lens {lens}: max row rel err {max(errs):.2e}", flush=True)
    assert max(errs) <= TOL


def test_dense_decode_deterministic_and_page_invariant():
    from paper_2607_24331_amd import dense_decode
    Hq, Hkv, d, lens = 8, 2, 128, [700, 300]
    pool, table, q = _case(Hq, Hkv, d, lens, seed=3, permute=False)
    args = (torch.from_numpy(q).cuda(), torch.from_numpy(pool).to(torch.bfloat16).cuda(),
            torch.from_numpy(table).cuda(), torch.tensor(lens, dtype=torch.int32).cuda(), 700, Hkv)
    a = dense_decode(*args, split_tokens=128).cpu().numpy()
    b = dense_decode(*args, split_tokens=128).cpu().numpy()
    assert np.array_equal(a, b)
    # move the pages and rewrite the table: bitwise the same
    perm = np.random.default_rng(1).permutation(pool.shape[0])
    pool2 = np.empty_like(pool)
    pool2[perm] = pool
    c = dense_decode(args[0], torch.from_numpy(pool2).to(torch.bfloat16).cuda(),
                     torch.from_numpy(perm[table].astype(np.int32)).cuda(), args[3], 700, Hkv,
                     split_tokens=128).cpu().numpy()
    assert np.array_equal(a, c)
