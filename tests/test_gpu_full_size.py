"""GPU path vs the CPU oracle on the full-size workloads, in the launch configuration
bench.py times (one cct_build, or cct_build + 32 cct_merge calls, on torch's current
stream): every output array compared element by element, bit-exact.

These are the largest parity cases (up to 72M events, 5.2G frames); each takes
tens of seconds, most of it the single-threaded oracle."""
import numpy as np
import pytest

import oracle
import tracegen
from gpu_util import assert_same, gpu_tree, node_paths, to_dev, torch_or_skip

pytestmark = [pytest.mark.gpu, pytest.mark.slow, pytest.mark.timeout(900)]


@pytest.fixture(autouse=True)
def _gpu():
    torch_or_skip()
    yield
    import torch
    import paper_2411_02797_amd as cct
    torch.cuda.synchronize()
    cct.release_cached_memory()
    torch.cuda.empty_cache()


@pytest.mark.parametrize("name", ["layered_16m", "deep_recursion"])
def test_full_size_build(name):
    # 16,777,216 events / 1.16G frames (M = 2), and 4,194,304 events / 1.59G frames of
    # depth 256..512 (M = 1)
    o, f, w = tracegen.generate(name)
    print(f"{name}: N={o.size - 1:,} F={f.size:,}", flush=True)
    got = gpu_tree(o, f, w)
    want = oracle.build_tree(o, f, w)
    assert_same(got, want, name)
    code, node = oracle.check(got, oracle.total_metrics(w))
    assert code == 0, f"{name}: invariant {oracle.CHECK_MESSAGES.get(code)} fails at node {node}"


def test_full_size_merge():
    # 8,388,608-event base, then 32 chunks of 2,097,152 events (20% from paths never
    # seen before the chunk, one full-range metric that wraps mod 2^64), merged one
    # at a time; equal to the oracle that ingested the same events
    import paper_2411_02797_amd as cct
    o, f, w = tracegen.generate("merge_base")
    orc = oracle.Oracle(w.shape[1])
    orc.ingest(o, f, w)
    tree = cct.build(*to_dev(o, f, w))
    total = oracle.total_metrics(w)
    for c in range(32):
        co, cf, cw = tracegen.generate("merge_chunk", chunk=c)
        orc.ingest(co, cf, cw)
        tree.merge(*to_dev(co, cf, cw))
        total = total + oracle.total_metrics(cw)
    got = tree.to_numpy()
    tree.free()
    want = orc.tree()
    orc.close()
    assert_same(got, want, "merge: 8M base + 32 x 2M chunks")
    code, node = oracle.check(got, total)
    assert code == 0, f"merge: invariant {oracle.CHECK_MESSAGES.get(code)} fails at node {node}"


def test_full_size_query():
    # cct_query over the full 16M-event tree: 20,000 sampled nodes (every depth) and
    # 1,000 absent paths; ids, exclusive and inclusive sums against the tree's arrays,
    # and 200 of the nodes against the oracle's scan of every event
    torch = torch_or_skip()
    import paper_2411_02797_amd as cct
    o, f, w = tracegen.generate("layered_16m")
    tree = cct.build(*to_dev(o, f, w))
    arr = tree.to_numpy()
    U = arr["parent"].size
    rng = np.random.default_rng(5)
    nodes = np.unique(np.concatenate([[0, U - 1], rng.integers(0, U, 20_000)]))
    paths = node_paths(arr, nodes)
    absent = [p + [int(x)] for p, x in zip(paths[:1000], rng.integers(0, 2**32, 1000, dtype=np.uint64))]
    qo = np.zeros(len(paths) + len(absent) + 1, np.int64)
    qo[1:] = np.cumsum([len(p) for p in paths + absent])
    qf = np.array([x for p in paths + absent for x in p], np.uint32)
    dev = torch.device("cuda", 0)
    ids, ex, inc = tree.query(torch.from_numpy(qo).to(dev), torch.from_numpy(qf.view(np.int32)).to(dev))
    ids, ex, inc = ids.cpu().numpy(), ex.cpu().numpy().view(np.uint64), inc.cpu().numpy().view(np.uint64)
    tree.free()
    n = nodes.size
    assert np.array_equal(ids[:n], nodes)
    assert np.array_equal(ex[:n], arr["excl"][nodes]) and np.array_equal(inc[:n], arr["incl"][nodes])
    # an appended random frame is absent unless that child exists (then it must be found)
    for j, p in enumerate(absent):
        if ids[n + j] != -1:
            v = int(ids[n + j])
            assert node_paths(arr, [v])[0] == p
    sample = nodes[rng.choice(n, 200, replace=False)]
    so = np.zeros(sample.size + 1, np.int64)
    sp = node_paths(arr, sample)
    so[1:] = np.cumsum([len(p) for p in sp])
    sf = np.array([x for p in sp for x in p], np.uint32)
    cnt, sex, sinc = oracle.point_query(o, f, w, so, sf)
    assert np.array_equal(sex, arr["excl"][sample]) and np.array_equal(sinc, arr["incl"][sample])
