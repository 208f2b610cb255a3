"""Host-side logic that needs no GPU: which parameters the optimiser step hands to Muon and
which to schedule-free AdamW, and the seeded inputs of the stack's two ends."""

import numpy as np
import pytest

from paper_2606_03681_amd import stack
from paper_2606_03681_amd import workloads as wl


@pytest.mark.parametrize("E,H,block", [(256, 768, "pre"), (192, 384, "post"), (64, 128, "post")])
def test_muon_matrices_and_adamw_segments_partition_the_layer(E, H, block):
    mats = stack.muon_matrices(E, H, block)
    total = wl.param_count(E, H, block)
    # Q, K, V of both attentions as E x E, both output projections, W1 [H][E], W2 [E][H]
    shapes = sorted((r, c) for _, r, c in mats)
    assert shapes == sorted([(E, E)] * 8 + [(H, E), (E, H)])
    segs = stack.adamw_segments(total, mats)
    cover = np.zeros(total, np.int32)
    for o, r, c in mats:
        cover[o:o + r * c] += 1
    for o, n in segs:
        cover[o:o + n] += 1
    assert np.all(cover == 1)
    # the AdamW segments are exactly the one-dimensional parameters (biases and norm weights)
    off, one_d = 0, 0
    for name, shape, kind in wl.param_layout(E, H, block):
        if len(shape) == 1:
            one_d += shape[0]
        off += int(np.prod(shape))
    assert sum(n for _, n in segs) == one_d


def test_adamw_segments_without_muon_cover_everything():
    assert stack.adamw_segments(1000, []) == [(0, 1000)]
    assert stack.adamw_segments(10, [(0, 2, 5)]) == []
    assert stack.adamw_segments(12, [(2, 1, 3)]) == [(0, 2), (5, 7)]


def test_ends_inputs_shapes_and_ranges():
    w = wl.make_workload("record9-bf16", with_dY=False, datasets=[0, 5])
    e = wl.make_ends_inputs(w)
    assert (e.G, e.offsets, e.T, e.K, e.mean) == (5, (0, 1, 3, 7, 12), 24, 10, True)
    assert e.x.shape == (2, 1000, 20) and e.labels.shape == (2, 1000)
    assert np.all(e.n_feat == 20)
    for b in range(2):
        assert 0 <= e.labels[b].min() and e.labels[b].max() < e.n_class[b] <= 10
        m = e.n_feat[b]
        assert e.cell_mask[b].tolist() == [1] * m + [0] * (20 - m) + [1]
    w2 = wl.make_workload(4, with_dY=False, datasets=[3])
    e2 = wl.make_ends_inputs(w2)
    assert e2.G == 1 and not e2.mean and e2.T == 0
    # the feature count follows the workload's prefix mask
    assert e2.n_feat[0] == int(w2.cell_mask[0][:-1].sum())


def test_ends_inputs_regenerate_per_dataset():
    """A dataset's ends inputs do not depend on which other datasets are generated."""
    a = wl.make_ends_inputs(wl.make_workload(4, with_dY=False, datasets=[1, 2]))
    b = wl.make_ends_inputs(wl.make_workload(4, with_dY=False, datasets=[2]))
    assert np.array_equal(a.x[1], b.x[0]) and np.array_equal(a.labels[1], b.labels[0])
    assert np.array_equal(a.params, b.params)
