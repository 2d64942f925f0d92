"""GPU test of the library-owned workspace: growing it neither waits for the
device nor disturbs results.

A decode call that needs more workspace than its stream holds allocates a
larger buffer and releases the old one in stream order; with a long stretch
of work already queued on the stream the call must return before that work
has finished (the stream still reports pending work), and every result --
the call queued before the growth, which still reads the old buffer, and the
calls after it -- must match the fp64 oracle.
"""
from __future__ import annotations

import math
import time

import numpy as np
import pytest
import torch

import oracle
from attn_inputs import random_bf16
from tests.gpu_common import announce, compare

pytestmark = pytest.mark.gpu

DEV = "cuda"


@pytest.fixture(scope="module")
def pa():
    import paper_2609_29219_amd as pa
    assert torch.cuda.is_available(), "GPU tests need a HIP device"
    return pa


def _decode_ref(q, k, v):
    B, H, d = q.shape
    Skv = k.shape[2]
    sc = float(np.float32(1.0 / math.sqrt(d)))
    return oracle.attn(q.reshape(B, H, 1, d).contiguous(), k, v, B, H, 1, Skv, d, sc,
                       False).reshape(B, H, d)


def test_workspace_growth_does_not_wait_for_queued_work(pa):
    stream = torch.cuda.Stream()  # a fresh stream: its workspace starts empty
    B, H, Skv, d = 4, 8, 3000, 128
    q = random_bf16((B, H, d), 1500)
    k, v = random_bf16((B, H, Skv, d), 1501), random_bf16((B, H, Skv, d), 1502)
    ref = _decode_ref(q, k, v)
    qd, kd, vd = q.to(DEV), k.to(DEV), v.to(DEV)
    M = 8192
    a = random_bf16((M, M), 1503).to(DEV)
    b = random_bf16((M, M), 1504).to(DEV)
    c = torch.empty((M, M), dtype=torch.float32, device=DEV)
    splits = (1, 16, 96)  # workspace B*H*n*(d+2)*4 bytes: 16 KiB, 266 KiB, 1.6 MiB
    for n in splits:  # plan every shape first (host work only), so the timed calls only launch
        pa.decode_workspace_bytes(B, H, H, Skv, d, n)
    pa.gemm_plan(M, M, M)
    torch.cuda.synchronize()
    with torch.cuda.stream(stream):
        announce("workspace: first decode on a fresh stream")
        outs = [pa.attn_decode(qd, kd, vd, n_splits=splits[0])]
        stream.synchronize()
        for n in splits[1:]:
            announce(f"workspace: growth to n_splits={n} behind queued GEMMs")
            for _ in range(12):  # ~12 ms of queued work
                pa.gemm(a, b, c)
            t0 = time.perf_counter()
            outs.append(pa.attn_decode(qd, kd, vd, n_splits=n))
            host_ms = (time.perf_counter() - t0) * 1e3
            pending = not stream.query()
            print(f"[workspace] growth call n_splits={n}: {host_ms:.3f} ms host time, "
                  f"stream still busy: {pending}", flush=True)
            assert pending, "the growing call waited for the queued work"
            assert host_ms < 5.0, f"the growing call took {host_ms:.2f} ms of host time"
        stream.synchronize()
    for n, o in zip(splits, outs):
        compare(o, ref, f"decode n_splits={n} around workspace growth")
