"""Randomized parity across the whole API: per seed, random sizes, alphabet, path lengths,
metric count (1..8), value ranges (small, full uint64, tiny), frame ids (small or over all of
uint32), some empty paths, with or without statistics; a build and up to three merges, some of
them activity flushes with repeated and unregistered IDs.  Every output is compared with the
oracle: tree arrays, statistics (integers bit-exact, mean and deviation within 4 ulp), the
bottom-up view, random filters and queries of sampled nodes and absent paths."""
import numpy as np
import pytest

import oracle
import tracegen
from gpu_util import csr, node_paths, to_dev, torch_or_skip

pytestmark = [pytest.mark.gpu, pytest.mark.slow]


@pytest.fixture(autouse=True)
def _gpu():
    torch_or_skip()


def u64(a):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, np.uint64).view(np.int64)).to(torch.device("cuda", 0))


def shape_values(rng, o, f, w):
    kind = rng.integers(0, 4)
    if kind == 1:
        w = rng.integers(0, 2**64, size=w.shape, dtype=np.uint64)
    elif kind == 2:
        w = (w % np.uint64(3)).astype(np.uint64)
    if rng.random() < 0.3 and f.size:
        f = (f.astype(np.uint64) * np.uint64(0x9E3779B1) % np.uint64(2**32)).astype(np.uint32)
    if rng.random() < 0.2 and o.size > 3:  # some empty paths: drop the frames of a few events
        keep = np.ones(o.size - 1, bool)
        keep[rng.integers(0, o.size - 1, max(1, (o.size - 1) // 20))] = False
        lens = np.diff(o) * keep
        no = np.zeros_like(o)
        np.cumsum(lens, out=no[1:])
        nf = np.concatenate([f[o[i]:o[i + 1]] for i in range(o.size - 1) if keep[i]] or [np.zeros(0, np.uint32)])
        o, f = no, nf.astype(np.uint32)
    return o, f, w


def check(seed):
    import torch

    import paper_2411_02797_amd as cct
    dev = torch.device("cuda", 0)
    rng = np.random.default_rng(seed)
    m = int(rng.integers(1, 9))
    n_ids = int(rng.choice([2, 10, 100, 3000, 60000]))
    max_len = int(rng.choice([1, 4, 16, 40, 130]))
    n0 = int(rng.choice([0, 1, 50, 3000, 40000]))
    stats = bool(rng.random() < 0.5)
    o, f, w = tracegen.random_paths(max(n0, 1), n_ids, max_len, m, seed=seed)
    if n0 == 0:
        o, f, w = np.zeros(1, np.int64), np.zeros(0, np.uint32), np.zeros((0, m), np.uint64)
    o, f, w = shape_values(rng, o, f, w)
    orc = oracle.Oracle(m, stats=stats)
    orc.ingest(o, f, w)
    events = [(o, f, w)]
    tree = cct.build(*to_dev(o, f, w), stats=stats)
    steps = ["build"]
    for k in range(int(rng.integers(0, 4))):
        o2, f2, w2 = tracegen.random_paths(int(rng.integers(1, 20000)), n_ids, max_len, m, seed=seed * 7 + k + 1)
        o2, f2, w2 = shape_values(rng, o2, f2, w2)
        if rng.random() < 0.4 and o2.size > 1:  # an activity flush: IDs, repeats, unregistered
            n = o2.size - 1
            ids = rng.permutation(10**7)[:n].astype(np.uint64) + np.uint64(rng.integers(0, 2**40))
            take = rng.random(n) < 0.9
            rec = np.concatenate([ids[take], ids[rng.integers(0, n, n // 5)], np.uint64(2**63) + np.arange(7, dtype=np.uint64)])
            rng.shuffle(rec)
            met = rng.integers(0, 2**62, size=(rec.size, m), dtype=np.uint64)
            to2, tf2, _ = to_dev(o2, f2, np.zeros((n, m), np.uint64))
            un = tree.merge_activity(to2, tf2, u64(ids), u64(rec), u64(met))
            bo, bf, bw, want_un = oracle.join_activity_calls(o2, f2, ids, rec, met)
            assert un == want_un, (un, want_un)
            orc.ingest(bo, bf, bw)
            events.append((bo, bf, bw))
            steps.append("activity")
        else:
            tree.merge(*to_dev(o2, f2, w2))
            orc.ingest(o2, f2, w2)
            events.append((o2, f2, w2))
            steps.append("merge")
    want = orc.tree()
    orc.close()
    got = tree.to_numpy()
    for k in ("parent", "frame", "depth", "excl", "incl"):
        assert np.array_equal(got[k], want[k]), k
    U = want["parent"].size
    if stats:
        st = tree.stats(device="cpu")
        for k in ("count_excl", "count_incl", "min_excl", "min_incl", "sumsq_excl", "sumsq_incl"):
            assert np.array_equal(st[k].numpy().view(np.uint64), want[k]), k
        nodes = rng.choice(U, min(U, 300), replace=False)
        d = oracle.derived_stats(want, nodes)
        for k, wv in d.items():
            g = st[k].numpy()[nodes]
            assert np.array_equal(np.isnan(g), np.isnan(wv)), k
            ok = np.isnan(wv) | (np.abs(g - wv) <= 4 * np.spacing(np.abs(np.nan_to_num(wv))))
            assert ok.all(), k
    # bottom-up view against the oracle's view of all events
    allo = [events[0][0]]
    for eo, _, _ in events[1:]:
        allo.append(allo[-1][-1] + eo[1:])
    ao = np.concatenate(allo)
    af = np.concatenate([e[1] for e in events])
    aw = np.concatenate([e[2] for e in events]).reshape(-1, m)
    v = tree.bottom_up(device="cpu")
    wf, wex, win = oracle.bottom_up(ao, af, aw)
    assert np.array_equal(v["frames"].numpy().view(np.uint32), wf)
    assert np.array_equal(v["excl"].numpy().view(np.uint64), wex)
    assert np.array_equal(v["incl"].numpy().view(np.uint64), win)
    # filters
    for _ in range(3):
        j = int(rng.integers(0, m))
        p, q = int(rng.integers(0, 2**64, dtype=np.uint64)), int(rng.integers(1, 2**64, dtype=np.uint64))
        if rng.random() < 0.5:
            p, q = int(rng.integers(0, 5)), int(rng.integers(1, 50))
        den = str(rng.choice(["one", "metric", "root"]))
        kw = dict(num_excl=bool(rng.random() < 0.5), den=den, den_metric=int(rng.integers(0, m)),
                  den_excl=bool(rng.random() < 0.5) and den == "metric", leaves_only=bool(rng.random() < 0.3))
        op = int(rng.choice([1, -1]))
        assert np.array_equal(tree.filter(j, op, p, q, **kw).cpu().numpy(), oracle.filter_nodes(want, j, op, p, q, **kw))
    # queries: sampled nodes and absent paths
    nodes = rng.choice(U, min(U, 200), replace=False)
    paths = node_paths(want, nodes) + [[0xFFFFFFFE, 3], [1] * 700]
    qo, qf = csr(paths)
    ids, ex, inc = tree.query(torch.from_numpy(qo).to(dev), torch.from_numpy(qf.view(np.int32)).to(dev))
    ids = ids.cpu().numpy()
    exp = list(nodes) + [-1, -1]
    # an "absent" path may exist in a tree with such frames: check it by the oracle's walk
    for t, pth in enumerate(paths[-2:]):
        hit = [v for v in range(U) if node_paths(want, [v])[0] == pth] if U < 5000 else []
        if hit:
            exp[len(nodes) + t] = hit[0]
    if U < 5000:
        assert np.array_equal(ids, np.array(exp)), "query ids"
    else:
        assert np.array_equal(ids[:len(nodes)], nodes), "query ids"
    assert np.array_equal(inc.cpu().numpy()[:len(nodes)].view(np.uint64), want["incl"][nodes])
    tree.free()
    return f"m={m} ids={n_ids} len<={max_len} n0={n0} stats={stats} {'+'.join(steps)} U={U}"


@pytest.mark.timeout(300)
@pytest.mark.parametrize("seed", range(40))
def test_random_configuration(seed):
    print(f"seed {seed}: {check(seed)}", flush=True)
