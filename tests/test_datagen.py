"""The seeded input generators: the per-tensor host generator gives the same values as the flat one."""
import numpy as np

from paper_2607_22614_amd import datagen, workloads


def test_named_tensors_equal_their_slices_of_the_flat_buffer():
    wl = workloads.TINY
    flat = datagen.make_flat_numpy(wl.model, wl.train_shards, 9)
    names = ["embed", "layers.0.q", "layers.1.ln2", "final_norm", "lm_head"]
    got = datagen.make_tensors_numpy(wl.model, 9, names, workers=3)
    assert set(got) == set(names)
    off = 0
    for name, numel, _ in datagen.tensor_list(wl.model):
        if name in got:
            assert np.array_equal(got[name].view(np.uint32), flat[off:off + numel].view(np.uint32)), name
        off += numel
