"""Host-side DGC pieces: the sparsity warm-up schedule and the argument
checks of bytecomp_compress_dgc (no device work)."""
import ctypes

import pytest

from paper_2205_14465_amd import binding as B
from paper_2205_14465_amd import dgc


def test_warmup_schedule_sparsities():
    # DGC's warm-up: 75%, 93.75%, 98.4375%, 99.6% sparsity, then the target
    dens = [dgc.warmup_ratio(e, 0.001) for e in range(6)]
    assert dens[:4] == [0.25, 0.0625, 0.015625, 0.00390625]
    assert dens[4:] == [0.001, 0.001]
    assert dgc.warmup_ratio(2, 0.05) == 0.05  # never below the final ratio


def test_compress_dgc_argument_errors():
    L = B.lib()
    t = (B.bc_tensor * 1)()
    t[0].grad = 0x1000
    t[0].residual = 0x2000
    t[0].n = 100
    t[0].dtype = 0
    vel = (ctypes.c_void_p * 1)(0x3000)
    pay = B.bc_payload(idx=0x4000, val=0x5000)
    ws = ctypes.c_void_p(0x6000)
    big = 1 << 30
    assert L.bytecomp_compress_dgc(3, 0.01, 0, 0.9, t, vel, 1, pay, ws, big, None) == -2  # sign: not sparse
    assert L.bytecomp_compress_dgc(4, 0.01, 0, 0.9, t, vel, 1, pay, ws, big, None) == -2
    assert L.bytecomp_compress_dgc(0, 0.01, 0, 0.9, t, None, 1, pay, ws, big, None) == -1
    assert L.bytecomp_compress_dgc(0, 0.01, 0, 0.9, t, vel, 0, pay, ws, big, None) == 0  # T = 0: no-op
    assert L.bytecomp_compress_dgc(0, 0.01, 0, 0.9, t, vel, 1, pay, None, big, None) == -7
    assert L.bytecomp_compress_dgc(0, 0.01, 0, 0.9, t, vel, 1, pay, ws, 16, None) == -7
    bad = (ctypes.c_void_p * 1)(0x3004)
    assert L.bytecomp_compress_dgc(0, 0.01, 0, 0.9, t, bad, 1, pay, ws, big, None) == -9
    nul = (ctypes.c_void_p * 1)(None)
    assert L.bytecomp_compress_dgc(0, 0.01, 0, 0.9, t, nul, 1, pay, ws, big, None) == -1
    t[0].residual = None
    assert L.bytecomp_compress_dgc(0, 0.01, 0, 0.9, t, vel, 1, pay, ws, big, None) == -1
