"""The all-core oracle (OpenMP over tensors and element ranges, used only
for the benchmark's CPU baseline) gives results bit-identical to the serial
oracle, for every kind, at several thread counts."""
import numpy as np
import pytest

import oracle as O

from .exact_ref import same_f32_arrays

KINDS = ("topk", "topk_sampled", "randk", "sign", "terngrad", "qsgd4", "qsgd8")


def _set(rng, ns, f16=False):
    grads = [(rng.standard_normal(n) * 10.0 ** rng.uniform(-3, -1)).astype(np.float16 if f16 else np.float32)
             for n in ns]
    resids = [(rng.standard_normal(n) * 1e-4).astype(np.float32) for n in ns]
    return grads, resids


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("threads", [1, 3, 8])
def test_omp_compress_and_aggregate_match_serial(kind, threads):
    rng = np.random.default_rng(60 + KINDS.index(kind))
    ns = [0, 1, 33, 4095, 4096, 4097, 12289, 70001, 5000]
    grads, resids = _set(rng, ns, f16=(kind == "sign"))
    want, want_e = O.compress_set(kind, 0.05, 9, grads, resids)
    got, got_e = O.compress_list_omp(kind, 0.05, 9, grads, resids, threads)
    for key in want:
        assert np.array_equal(np.asarray(got[key]).view(np.uint8), np.asarray(want[key]).view(np.uint8)), key
    for a, b in zip(got_e, want_e):
        assert np.array_equal(a.view(np.uint32), b.view(np.uint32))
    # aggregate of W payloads (compressions of perturbed gradients)
    pays = [want]
    for w in range(1, 5):
        g2 = [(g.astype(np.float32) * np.float32(1 + 0.1 * w)).astype(g.dtype) for g in grads]
        pays.append(O.compress_set(kind, 0.05, 9 + w, g2, None)[0])
    ref = O.aggregate_set(kind, ns, pays, 0.25)
    out = O.aggregate_list_omp(kind, ns, pays, 0.25, threads)
    for a, b in zip(out, ref):
        assert same_f32_arrays(a, b)


def test_omp_reports_threads():
    assert O.omp_max_threads() >= 1
