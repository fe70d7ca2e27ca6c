"""Shared helpers of the test suite: small model builders and the error metric."""
import numpy as np

import synth

# Shrunken variants of the five workloads: every kernel path of the full-size
# model, several tiles and a ragged tail, and a CPU oracle that finishes in
# seconds.
SMALL = {
    1: dict(hw=16),
    2: dict(batch=2, hw=64, blocks=(1, 2, 2, 1), widths=(16, 32, 32, 64), n_cls=37),
    3: dict(batch=2, hw=64, arch=(16, "M", 32, "M", 64, 64, "M", 64, "M", 128, "M"), fc=(200, 96), n_cls=37,
            cut_after_pools=(3, 5)),
    4: dict(batch=2, seq=40, layers=3, hidden=128, heads=2, ffn=256, vocab=300, max_pos=64, slice_every=1),
    5: dict(batch=3, seq=9, hidden=64, emb=64, vocab=301),
    6: dict(batch=3, hw=32),
    7: dict(batch=3, hw=16),
}


def rel_err(got, ref):
    """max |got - ref| / max |ref| over the tensor (the per-tensor relative error)."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref, dtype=np.float64)
    den = np.abs(ref).max()
    return float(np.abs(got - ref).max() / (den if den > 0 else 1.0))


TOL = {"f32": 1e-4, "bf16": 2e-2}


def codec_ratio(c):
    """Compression ratio of a boundary of C channels: R = 8, the smallest ratio the paper
    studies, when it divides C (the code then has C / 8 channels), else the largest of 4 and
    2 that does, else 1."""
    return next((r for r in (8, 4, 2) if c % r == 0), 1)


def codec_ratios(model, cuts):
    """Compression ratio per cut (the boundary tensor leaving each cut node)."""
    return [codec_ratio(synth.boundary_channels(model, li)) for li in cuts]


def boundary_codecs(model, cuts, kind="ae"):
    """Boundary tensors of the cuts (every tensor crossing each cut, cut-major, ascending id)
    and AE codec weights for each, at codec_ratio of its channel count."""
    import oracle
    tids = [t for c in cuts for t in oracle.crossing_tensors(model, c)]
    ratios = [codec_ratio(synth.tensor_channels(model, t)) for t in tids]
    if kind != "ae" or not tids:
        return tids, None
    return tids, synth.make_codec_weights(model, cuts, ratio=ratios, tensors=tids)
