"""Fills a replay table with a workload's generated trajectories.

The rows are generated on the GPU chunk by chunk (gen_gpu.hip) into
staging tensors and handed, in insertion order, to a caller-supplied insert
function, so this module never calls the replay library itself.  Torch is
used only for device memory and the stream.
"""
import numpy as np
import torch

from . import fill_rows_gpu, insert_priorities


def fill_table(w, insert, device=0, chunk_bytes=1 << 30, stream=None):
    """insert(nrows, [device pointer per column], priorities uint32[nrows])
    is called once per chunk, in order, on `stream` (torch's current stream
    of `device` by default).  Returns the number of rows inserted."""
    dev = torch.device("cuda", device)
    stream = stream or torch.cuda.current_stream(dev)
    row_bytes = w.T * sum(w.elem_bytes)
    rows = w.n_insert if row_bytes == 0 else max(1, min(w.n_insert, chunk_bytes // row_bytes))
    staging = [torch.empty(rows * w.T * c.elem_bytes, dtype=torch.uint8, device=dev) for c in w.columns]
    keep = []
    k = 0
    while k < w.n_insert:
        n = min(rows, w.n_insert - k)
        for ci, c in enumerate(w.columns):
            fill_rows_gpu(c, ci, w.seed, w.T, k, n, staging[ci].data_ptr(), stream.cuda_stream)
        prio = insert_priorities(w.prio, w.seed, k, n)
        keep.append(prio)
        insert(n, [s.data_ptr() for s in staging], prio)
        k += n
    stream.synchronize()
    del keep
    return k
