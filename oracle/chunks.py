"""Reference rule for grouping a model's weights into transfer chunks (oracle).

Test infrastructure only. Paper Sec. 4.3 ("Model swapping and pipeline execution"):
parameters are grouped for transfer; groups that are too small cost synchronisation,
groups that are too large hurt the pipeline, and the group size is the "elbow" of
transfer throughput versus size (about 2 MB on the paper's testbed), found by profiling.

Reading: tensors are visited in first-use order; a chunk accumulates whole layers (a
layer is never split) and is closed at the first layer boundary where it holds at
least ``min_bytes``. Chunks tile the host buffer: chunk 0 starts at byte 0, every later
chunk starts at the offset of its first tensor, and the last one ends at the buffer end.

With ``per_tensor`` the unit is a tensor instead of a layer, which is the paper's own
model-agnostic grouping of parameters; with ``min_bytes = 0`` every tensor is a transfer
of its own, the parameter-level pipeline of the Sec. 6.1 breakdown.
"""
from __future__ import annotations


def plan(tensors, total_bytes: int, min_bytes: int, per_tensor: bool = False):
    """tensors: iterable of (layer, offset, nbytes) in first-use order.

    Returns a list of dicts {begin, end, first_layer, last_layer}.
    """
    layers = []                      # (layer, first offset, end offset) of each unit
    for layer, off, nb in tensors:
        if layers and layers[-1][0] == layer and not per_tensor:
            layers[-1][2] = off + nb
        else:
            layers.append([layer, off, off + nb])
    chunks = []
    cur = None
    for layer, off, end in layers:
        if cur is None:
            cur = {"begin": 0 if not chunks else off, "end": end, "first_layer": layer, "last_layer": layer}
        else:
            cur["end"], cur["last_layer"] = end, layer
        if cur["end"] - cur["begin"] >= min_bytes:
            chunks.append(cur)
            cur = None
    if cur is not None:
        chunks.append(cur)
    for a, b in zip(chunks, chunks[1:]):
        a["end"] = b["begin"]
    chunks[-1]["end"] = total_bytes
    return chunks
