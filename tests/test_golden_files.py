"""Consistency of the stored noise profiles (tests/golden/small_100_noise_profile.json and
mid_10_noise_profile.json, written by make_noise_profile.py from oracle runs only), which the
full-size GPU trajectory tests hold their later free-running points against.  CPU only: reads the
JSON, runs nothing."""
import json
import os

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _profile(name="small_100"):
    with open(os.path.join(GOLDEN, f"{name}_noise_profile.json")) as f:
        return json.load(f)


def test_injected_noise_has_the_stated_size():
    # at steps 0 and 1 the perturbed run still has the clean weights x_0 (the first update consumes
    # g_0 at t = 1), so the stored gradients differ by the injected noise alone: 1.2 % norm-wise for
    # both kinds (relative: each element times 1 + eps xi; additive: eps rms xi)
    p = _profile()
    assert p["grad_noise"] == 0.012
    for kind in ("relative", "additive"):
        for point in ("g@0", "g@1"):
            assert abs(p[kind][point]["median"] - 0.012) < 0.0006, (kind, point, p[kind][point])
        # the outputs of steps 0 and 1 are computed before any update: identical
        for point in ("y@0", "y@1"):
            assert p[kind][point]["max"] == 0.0, (kind, point)


def test_first_adam_update_is_insensitive_to_sign_preserving_noise():
    # Adam's first update is lr sign(g) (m / sqrt(v) = g / |g| up to the epsilon), so noise that keeps
    # every sign leaves it, and the Error Feedback buffer holding it, almost unchanged, while noise
    # that flips the signs of a tensor's smallest elements moves it by a tenth
    p = _profile()
    assert p["relative"]["u_prev@2"]["median"] < 1e-3
    assert p["additive"]["u_prev@2"]["median"] > 5e-2


def test_perturbed_runs_separate_over_the_iterations():
    # the separation the GPU test compares against grows with the iterations, for every stored
    # quantity, under both kinds of noise
    p = _profile()
    for kind in ("relative", "additive"):
        for q in ("x", "m", "v", "u_prev"):
            meds = [p[kind][f"{q}@{k}"]["median"] for k in (10, 50, 100)]
            assert meds[0] < meds[1] < meds[2], (kind, q, meds)


def test_mid_profile_injected_noise():
    # the mid workload's perturbed run (additive noise only): the same size at steps 0 and 1, no
    # output change before the first update, and the weights and momentum separating from step 3
    # to step 10
    p = _profile("mid_10")["additive"]
    for point in ("g@0", "g@1"):
        assert abs(p[point]["median"] - 0.012) < 0.0006, (point, p[point])
    for point in ("y@0", "y@1"):
        assert p[point]["max"] == 0.0, point
    for q in ("x", "m"):
        assert p[f"{q}@3"]["median"] < p[f"{q}@10"]["median"], q
