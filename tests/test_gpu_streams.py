"""Searches on one index issued back to back on two streams (each stream has
its own workspace, and for the partitioned search its own probe buffer):
every result equals the one computed alone on the default stream, bit for
bit, for the single-tile scan, the shared-key scan and the tiled
contraction, and for the partitioned search."""
import pytest
import torch

pytestmark = pytest.mark.gpu
DEV = "cuda:0"


def _keys(N, d, dt, seed):
    gen = torch.Generator(device="cuda").manual_seed(seed)
    x = torch.randn(N, d, device=DEV, generator=gen)
    x = (x / x.norm(dim=1, keepdim=True)).to(dt)
    cont = torch.randint(0, 32000, (N, 3), device=DEV, generator=gen, dtype=torch.int32)
    q = torch.randn(256, d, device=DEV, generator=gen)
    q = (q / q.norm(dim=1, keepdim=True)).contiguous()
    return x, cont, q


@pytest.mark.parametrize("N,d,dt,batches,k", [
    (40000, 256, torch.float16, (1, 64), 16),     # single-tile and shared-key scans
    (20011, 2048, torch.bfloat16, (1, 48), 10),   # single-tile scan and tiled contraction
], ids=["d256", "d2048"])
def test_two_streams_match_serial(gpu_lib, N, d, dt, batches, k):
    from paper_2502_15572_amd import Index
    x, cont, q = _keys(N, d, dt, N + d)
    ix = Index(x, cont)
    qs = [q[:B].contiguous() for B in batches]
    refs = [[t.clone() for t in ix.search(qq, k)] for qq in qs]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = [[], []]
    for _ in range(6):
        for i, s in enumerate(streams):
            with torch.cuda.stream(s):
                outs[i].append(ix.search(qs[i], k, stream=s))
    torch.cuda.synchronize()
    for i in range(2):
        for got in outs[i]:
            for a, b in zip(got, refs[i]):
                assert torch.equal(a, b)
    ix.close()


def test_partitioned_two_streams_match_serial(gpu_lib):
    from paper_2502_15572_amd import PartitionedIndex, kmeans_assign, train_partitions
    x, cont, q = _keys(30000, 64, torch.float16, 5)
    cents, _ = train_partitions(x, 32, iters=3, seed=1)
    ix = PartitionedIndex(x, cont, cents, kmeans_assign(x, cents))
    k, nprobe = 20, 6
    qs = [q[:3].contiguous(), q[3:40].contiguous()]
    refs = [[t.clone() for t in ix.search(qq, k, nprobe)] for qq in qs]
    torch.cuda.synchronize()
    streams = [torch.cuda.Stream(), torch.cuda.Stream()]
    outs = [[], []]
    for _ in range(6):
        for i, s in enumerate(streams):
            with torch.cuda.stream(s):
                outs[i].append(ix.search(qs[i], k, nprobe, stream=s))
    torch.cuda.synchronize()
    for i in range(2):
        for got in outs[i]:
            for a, b in zip(got, refs[i]):
                assert torch.equal(a, b)
    ix.close()
