"""Parity of the GPU draft assembly (Section 3.6) with the oracle: bit-exact
(integer work).  Hand-derived fixtures, random token matrices with many
repeats (small vocabulary), EOS inside drafts, k = DRESD_K_MAX, and the
padding ranks of a filtered search."""
import json
import os

import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
FIX = os.path.join(os.path.dirname(__file__), "golden", "draft_packing.json")


def gpu_pack(t, r, length, eos):
    from paper_2502_15572_amd import pack_drafts
    d, n = pack_drafts(torch.as_tensor(np.ascontiguousarray(t, np.int32)).to(DEV), r, length, eos)
    torch.cuda.synchronize()
    return d.cpu().numpy(), n.cpu().numpy()


def test_drafts_golden(gpu_lib):
    for c in json.load(open(FIX))["cases"]:
        d, n = gpu_pack(np.asarray(c["tokens"]), c["r"], c["length"], c["eos"])
        assert d.tolist() == c["drafts"], c["name"]
        assert n.tolist() == c["count"], c["name"]


CASES = [
    # (B, k, L, r, length, vocab, eos)
    (4, 10, 10, 10, 10, 3, 0),
    (7, 100, 10, 20, 8, 4, 0),
    (3, 1024, 6, 300, 3, 5, 1),
    (2, 33, 20, 3, 20, 2, 0),
    (64, 32, 10, 32, 10, 50, 0),
    (5, 16, 1, 16, 1, 3, 0),          # one-token values
    (2, 1, 4, 1, 4, 2, 1),            # one retrieved continuation
]


@pytest.mark.parametrize("B,k,L,r,length,vocab,eos", CASES,
                         ids=["B%d-k%d-L%d-r%d-len%d-v%d-eos%d" % c for c in CASES])
def test_drafts_parity(gpu_lib, B, k, L, r, length, vocab, eos):
    print("drafts", B, k, L, r, length, vocab, eos, flush=True)
    rng = np.random.default_rng(B * 1000 + k)
    t = rng.integers(0, vocab, (B, k, L)).astype(np.int32)
    want_d, want_n = oracle.pack_drafts(t, r, length, eos)
    d, n = gpu_pack(t, r, length, eos)
    assert np.array_equal(n, want_n)
    assert np.array_equal(d, want_d)


def test_drafts_after_filtered_search(gpu_lib):
    """Padding ranks of a filtered search (zero tokens) are dropped; the
    drafts all start with the query's next token."""
    from paper_2502_15572_amd import Index, pack_drafts
    rng = np.random.default_rng(3)
    N, d, L = 4000, 64, 6
    x = rng.standard_normal((N, d))
    x = torch.from_numpy((x / np.linalg.norm(x, axis=1, keepdims=True)).astype(np.float16)).to(DEV)
    cont = torch.from_numpy(rng.integers(1, 40, (N, L)).astype(np.int32)).to(DEV)
    q = torch.from_numpy(rng.standard_normal((3, d)).astype(np.float32)).to(DEV)
    q = q / q.norm(dim=1, keepdim=True)
    nt = torch.tensor([5, 7, 10 ** 6], dtype=torch.int32, device=DEV)
    ix = Index(x, cont)
    _, _, tok = ix.search(q, 200, next_tok=nt)
    drafts, count = pack_drafts(tok, 50, 4)
    want_d, want_n = oracle.pack_drafts(tok.cpu().numpy(), 50, 4)
    assert np.array_equal(drafts.cpu().numpy(), want_d) and np.array_equal(count.cpu().numpy(), want_n)
    assert count[2].item() == 0
    for b in range(2):
        assert (drafts[b, : count[b], 0] == nt[b]).all()
    ix.close()
