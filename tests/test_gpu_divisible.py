"""Divisible scheme on the GPU against the oracle: packing part j of a
payload, aggregating one part from W senders (ragged entry counts for the
sparse kinds), and the whole node-j step followed by the second
compression and the final decompress (paper Sec. 3.1, Reason #2)."""
import numpy as np
import pytest

import oracle as O
from tests.helpers import bits, torch_dev

pytestmark = pytest.mark.gpu

SEED = 14465


def _bounds(rng, ns, P, empty_part=False):
    out = []
    for n in ns:
        inner = sorted(int(x) * 32 for x in rng.integers(0, n // 32 + 1, size=P - 1))
        if empty_part and P > 2:
            inner[1] = inner[0]  # part 1 is empty
        out.append([0] + inner + [n])
    return out


WORD_KINDS = ("sign", "terngrad", "qsgd4", "qsgd8")


def _dev_payload(kind, p):
    if kind in WORD_KINDS:
        return {"bits": torch_dev(p["bits"].view(np.int32)), "scale": torch_dev(p["scale"])}
    return {"idx": torch_dev(p["idx"].view(np.int32)), "val": torch_dev(p["val"])}


def _oracle_payloads(kind, ratio, ns, W, rng):
    pays = []
    for w in range(W):
        grads = [(rng.standard_normal(n) * 0.01).astype(np.float32) for n in ns]
        pays.append(O.compress_set(kind, ratio, SEED + w, grads, None)[0])
    return pays


def _gpu_pack(kind, ratio, ns, dev_pay, bounds, j):
    import torch
    from paper_2205_14465_amd import binding as B
    out = B.alloc_payload(kind, ratio, ns)
    po = torch.full((len(ns) + 1,), -1, dtype=torch.int64, device="cuda")
    B.bytecomp_pack_part(kind, ratio, ns, dev_pay, bounds, j, out, po)
    torch.cuda.synchronize()
    return out, po


@pytest.mark.parametrize("kind", ["topk", "randk", "sign", "terngrad", "qsgd4", "qsgd8"])
@pytest.mark.parametrize("empty_part", [False, True])
def test_pack_part_matches_oracle(kind, empty_part):
    rng = np.random.default_rng(41 + empty_part)
    ns = [1, 31, 32, 100, 4097, 70000, 0, 250001]
    ratio = 0.05
    pay = _oracle_payloads(kind, ratio, ns, 1, rng)[0]
    dev = _dev_payload(kind, pay)
    P = 4
    bounds = _bounds(rng, ns, P, empty_part)
    for j in range(P):
        out, po = _gpu_pack(kind, ratio, ns, dev, bounds, j)
        want = O.pack_part_set(kind, ns, pay, bounds, j)
        got_off = po.cpu().numpy()
        assert np.array_equal(got_off, want["off"]), (j, got_off, want["off"])
        tot = int(want["off"][-1])
        if kind in WORD_KINDS:
            assert np.array_equal(out["bits"].cpu().numpy().view(np.uint32)[:tot], want["bits"]), j
            assert np.array_equal(bits(out["scale"].cpu().numpy()[:len(ns)]), bits(want["scale"]))
        else:
            assert np.array_equal(out["idx"].cpu().numpy().view(np.uint32)[:tot], want["idx"]), j
            assert np.array_equal(bits(out["val"].cpu().numpy()[:tot]), bits(want["val"])), j


@pytest.mark.parametrize("kind", ["topk", "randk", "sign", "terngrad", "qsgd4", "qsgd8"])
@pytest.mark.parametrize("W", [1, 3, 16, 64])
def test_aggregate_part_matches_oracle(kind, W):
    import torch
    from paper_2205_14465_amd import binding as B
    rng = np.random.default_rng(100 + W)
    ns = [33, 4096, 20001, 0, 150000]
    ratio = 0.02
    pays = _oracle_payloads(kind, ratio, ns, W, rng)
    P = 3
    bounds = _bounds(rng, ns, P, empty_part=(W == 3))
    whole = O.aggregate_set(kind, ns, pays, 1.0 / W)
    for j in range(P):
        lens = [b[j + 1] - b[j] for b in bounds]
        dev_parts, offs = [], []
        for p in pays:
            out, po = _gpu_pack(kind, ratio, ns, _dev_payload(kind, p), bounds, j)
            dev_parts.append(out)
            offs.append(po)
        outs = [torch.full((max(n, 1),), float("nan"), dtype=torch.float32, device="cuda")[:n] for n in lens]
        ws = B.alloc_workspace(kind, ratio, lens, W)
        B.bytecomp_aggregate_part(kind, ratio, dev_parts, None if kind in WORD_KINDS else offs, lens, outs,
                                  1.0 / W, ws)
        torch.cuda.synchronize()
        want_parts = O.aggregate_part_set(kind, lens, [O.pack_part_set(kind, ns, p, bounds, j) for p in pays],
                                          1.0 / W)
        for t in range(len(ns)):
            got = outs[t].cpu().numpy()
            assert np.array_equal(bits(got), bits(want_parts[t])), (j, t)
            lo, hi = bounds[t][j], bounds[t][j + 1]
            assert np.array_equal(bits(got), bits(whole[t][lo:hi])), (j, t)
        assert B.bytecomp_device_status(ws) == 0


def test_aggregate_part_large_tiles():
    # parts totalling at least 2^24 elements at low density take the
    # 8192-element tiles with ragged entry counts
    import torch
    from paper_2205_14465_amd import binding as B
    rng = np.random.default_rng(8)
    ns = [(1 << 25) + 4100, 3000]
    ratio = 0.005
    W = 12
    off = O.sparse_offsets(ns, ratio)
    pays = []
    for w in range(W):
        idx = [np.sort(rng.choice(n, size=int(O.k_for(n, ratio)), replace=False)).astype(np.uint32) for n in ns]
        val = [rng.standard_normal(i.size).astype(np.float32) for i in idx]
        pays.append({"idx": np.concatenate(idx), "val": np.concatenate(val), "off": off})
    P = 2
    bounds = [[0, (n // 2) // 32 * 32, n] for n in ns]
    j = 0
    lens = [b[j + 1] - b[j] for b in bounds]
    assert sum(lens) >= 1 << 24
    dev_parts, offs = [], []
    for p in pays:
        out, po = _gpu_pack("topk", ratio, ns, _dev_payload("topk", p), bounds, j)
        dev_parts.append(out)
        offs.append(po)
    outs = [torch.full((n,), float("nan"), dtype=torch.float32, device="cuda") for n in lens]
    ws = B.alloc_workspace("topk", ratio, lens, W)
    B.bytecomp_aggregate_part("topk", ratio, dev_parts, offs, lens, outs, 1.0 / W, ws)
    torch.cuda.synchronize()
    want = O.aggregate_part_set("topk", lens, [O.pack_part_set("topk", ns, p, bounds, j) for p in pays], 1.0 / W)
    for t in range(len(ns)):
        assert np.array_equal(bits(outs[t].cpu().numpy()), bits(want[t])), t
    assert B.bytecomp_device_status(ws) == 0


@pytest.mark.parametrize("kind", ["topk", "sign", "terngrad", "qsgd8"])
def test_divisible_step_end_to_end(kind):
    """Node j's step for every j: aggregate the parts, compress the aggregate
    again (no error feedback), and decompress every node's result into the
    full tensors; the oracle composes the same definitions."""
    import torch
    from paper_2205_14465_amd import binding as B
    rng = np.random.default_rng(7)
    ns = [4096 * 3 + 17, 64, 90000]
    W, P, ratio = 8, 4, 0.05
    pays = _oracle_payloads(kind, ratio, ns, W, rng)
    bounds = _bounds(rng, ns, P)
    finals = [torch.full((n,), float("nan"), dtype=torch.float32, device="cuda") for n in ns]
    want_finals = [np.zeros(n, np.float32) for n in ns]
    for j in range(P):
        lens = [b[j + 1] - b[j] for b in bounds]
        dev_parts, offs = [], []
        for p in pays:
            out, po = _gpu_pack(kind, ratio, ns, _dev_payload(kind, p), bounds, j)
            dev_parts.append(out)
            offs.append(po)
        slices = [torch.empty(max(n, 1), dtype=torch.float32, device="cuda")[:n] for n in lens]
        ws = B.alloc_workspace(kind, ratio, lens, W)
        B.bytecomp_aggregate_part(kind, ratio, dev_parts, None if kind in WORD_KINDS else offs, lens, slices,
                                  1.0 / W, ws)
        # second compression of node j's aggregate (no residual)
        sec = B.alloc_payload(kind, ratio, lens)
        ws2 = B.alloc_workspace(kind, ratio, lens, 1)
        B.bytecomp_compress(kind, ratio, SEED, slices, None, sec, ws2)
        # every node decompresses node j's payload into the full tensors
        views = [finals[t][bounds[t][j]:bounds[t][j + 1]] for t in range(len(ns))]
        ws3 = B.alloc_workspace(kind, ratio, lens, 1)
        B.bytecomp_decompress_aggregate(kind, ratio, [sec], lens, views, 1.0, ws3)
        torch.cuda.synchronize()
        # oracle
        agg = O.aggregate_part_set(kind, lens, [O.pack_part_set(kind, ns, p, bounds, j) for p in pays], 1.0 / W)
        sec_o, _ = O.compress_set(kind, ratio, SEED, agg, None)
        dec = O.aggregate_set(kind, lens, [sec_o], 1.0)
        for t in range(len(ns)):
            want_finals[t][bounds[t][j]:bounds[t][j + 1]] = dec[t]
    for t in range(len(ns)):
        got = finals[t].cpu().numpy()
        # sign: the second compression's scales are fp64 sums in different
        # orders on the two sides, equal in practice at these sizes
        assert np.array_equal(bits(got), bits(want_finals[t])), t
