"""The seeded input generator against the published SplitMix64 definition."""
import numpy as np
import torch

import synth

# First outputs of Vigna's reference splitmix64.c seeded with x = 1234567.
REF_1234567 = [6457827717110365317, 3203168211198807973, 9817491932198370423,
               4593380528125082431, 16408922859458223821]


def test_splitmix64_reference_vector():
    s, got = 1234567, []
    for _ in range(5):
        s, o = synth.splitmix64_scalar(s)
        got.append(o)
    assert got == REF_1234567
    vec = synth.raw64(1234567, 0, 5)
    assert [int(v) & synth.M64 for v in vec] == REF_1234567


def test_irwin_hall_moments_and_bounds():
    w = synth.irwin_hall(synth.stream_key(0, 12345), 1 << 20, 0.02).double()
    assert abs(w.mean().item()) < 1e-4
    assert abs(w.std().item() - 0.02) < 2e-4
    assert w.abs().max().item() <= 0.02 * 3.4642


def test_tokens_uniform_and_exclude_mask():
    t = synth.uniform_tokens(synth.stream_key(1, 3), 200000, 100)
    assert int(t.min()) == 0 and int(t.max()) == 98
    counts = torch.bincount(t, minlength=99).double()
    assert (counts.std() / counts.mean()).item() < 0.05


def test_streams_differ_and_repeat():
    a = synth.layer_weights(synth.config("tiny"), 0)
    b = synth.layer_weights(synth.config("tiny"), 0)
    c = synth.layer_weights(synth.config("tiny"), 1)
    assert torch.equal(a["wq"], b["wq"]) and not torch.equal(a["wq"], c["wq"])
    assert not torch.equal(a["wq"][:8, :8], a["wk"][:8, :8])
