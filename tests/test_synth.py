"""The input generator: determinism, exact storage rounding, workload shapes."""
import numpy as np
import torch

import synth


def test_bf16_round_is_torch_round_to_nearest_even():
    r = np.random.default_rng(0)
    x = np.concatenate([r.standard_normal(100000).astype(np.float32),
                        np.array([1 + 2 ** -8, 1 + 3 * 2 ** -8, -1 - 2 ** -8, 0.0, -0.0,
                                  np.inf, -np.inf], dtype=np.float32)])
    ours = synth.bf16_round(x)
    ref = torch.from_numpy(x).to(torch.bfloat16).to(torch.float32).numpy()
    assert np.array_equal(ours.view(np.uint32), ref.view(np.uint32))
    # exactly representable: a second rounding is the identity
    assert np.array_equal(synth.bf16_round(ours).view(np.uint32), ours.view(np.uint32))


def test_streams_are_per_sample_and_deterministic():
    w = synth.workload(3)
    a = synth.sample_activations(w, 0, 5)
    b = synth.layer_activations(w, 0, samples=[4, 5])
    assert np.array_equal(a["h"], b["h"][1]) and np.array_equal(a["v"], b["v"][1])
    assert not np.array_equal(b["h"][0], b["h"][1])
    w4 = synth.workload(4)
    assert not np.array_equal(synth.layer_weights(w4, 0)["W1"][:4, :64],
                              synth.layer_weights(w4, 1)["W1"][:4, :64])


def test_workload_shapes():
    w = synth.workload(2)
    assert (w.T, w.ds, w.router_in) == (305, 16, 8320)
    assert synth.workload(4).T == 177 and synth.workload(5).T == 2048 and synth.workload(5).ds == 4
    assert list(np.bincount(w.types(), minlength=4)) == [256, 48, 1, 0]
    s = synth.sample_scores(synth.workload(5), 0, 0)
    assert s.dtype == np.float32 and s.shape == (2048, 32)
