"""Digests of the hot path's outputs over whole demand streams.

The 64-rank workload plans a stream of 100 demand matrices and the 256-rank
workload a stream of 1000; parity over these streams is checked through
SHA-256 digests that the oracle wrote once (``golden/make_stream_digests.py``)
and the GPU path must reproduce:

  demand     the N x N int64 byte-demand matrix
  schedule   K, tau and the family, destination, instance and bytes of every
             lane of every step
  send       every SAMPLE_STRIDE-th byte of rank 0's send buffer (a prime
             stride, so every byte position of a row is sampled somewhere),
             with the buffer's length
  step_off   the K + 1 step offsets of that send buffer

This module holds hashing and the seeded routing generation for worker
processes only; none of the method's arithmetic.
"""
from __future__ import annotations

import hashlib
import os
import sys

import numpy as np

SAMPLE_STRIDE = 4099
# the matrices in stream_digests.json: every matrix of the 64-rank stream,
# every 10th of the 256-rank stream (all 1000 are in stream_digests_256_all.json,
# which the GPU suite checks)
STREAMS = {3: list(range(100)), 5: list(range(0, 1000, 10))}
GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "stream_digests.json")
# every matrix of the 256-rank stream
GOLDEN_ALL5 = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "stream_digests_256_all.json")
# the first matrix of the 256-rank workload planned on nodes with cross-socket
# peer to peer (SYS paths)
GOLDEN_SYS256 = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "sys256_digest.json")
# the planner's largest shape: 1,024 ranks (128 nodes) under the hot-destination
# demand of vpgen.hot_destinations_demand, k_max = 32N
GOLDEN_1024 = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden", "plan1024_digest.json")


def _sha(*arrays) -> str:
    h = hashlib.sha256()
    for a in arrays:
        h.update(np.ascontiguousarray(a).tobytes())
    return h.hexdigest()[:32]


def demand_digest(D) -> str:
    return _sha(np.asarray(D, dtype=np.int64))


def schedule_digest(s: dict) -> str:
    K = int(s["K"])
    return _sha(np.array([K, int(s["tau"])], np.int64),
                np.asarray(s["family"], np.int32)[:K], np.asarray(s["dst"], np.int32)[:K],
                np.asarray(s["inst"], np.int32)[:K], np.asarray(s["bytes"], np.int64)[:K])


def send_sample(send: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(send[::SAMPLE_STRIDE], dtype=np.uint8)


def send_digest(sample: np.ndarray, length: int) -> str:
    return _sha(np.array([length], np.int64), np.asarray(sample, np.uint8))


def step_off_digest(step_off) -> str:
    return _sha(np.asarray(step_off, np.int64))


def routing_job(args):
    """(config, matrix) -> (matrix, int32 [N, T, k] routing); for process pools."""
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    if root not in sys.path:
        sys.path.insert(0, root)
    import vpgen
    cid, m = args
    return m, vpgen.routing_all(vpgen.config(cid), m)


def pool_size() -> int:
    return max(1, min(12, (os.cpu_count() or 2) - 1))
