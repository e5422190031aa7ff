"""The device-side mesh generators (run here on the CPU through torch) follow
the host recipe: volume points lie in the box and outside the body, surface
points lie on the body, features are layer-normalised per point, chunks are
reproducible and independent of each other."""
import numpy as np
import torch

from ts3_synth import geometry as G
from ts3_synth.device_gen import DeviceSurface, DeviceVolume


def _radius(body, u):
    return body.radius(u)


def test_surface_points_lie_on_the_body_and_chunks_are_reproducible():
    d = DeviceSurface(3, 64, device="cpu", dtype=torch.float32)
    p = d.points(0, 4000).numpy()
    body = G.CarBody()
    r = p - np.asarray(G.BODY_CENTRE)
    dist = np.linalg.norm(r, axis=1)
    np.testing.assert_allclose(dist, _radius(body, r / dist[:, None]), rtol=1e-10)
    np.testing.assert_array_equal(d.points(0, 4000).numpy(), p)
    assert not np.array_equal(d.points(1, 4000).numpy(), p)


def test_volume_points_lie_in_the_box_outside_the_body():
    d = DeviceVolume(5, 64, device="cpu", dtype=torch.float32)
    p = d.points(0, 4000).numpy()
    lo, hi = np.asarray(G.VOLUME_BOX_LO), np.asarray(G.VOLUME_BOX_HI)
    assert ((p >= lo) & (p <= hi)).all()
    body = G.CarBody()
    r = p - np.asarray(G.BODY_CENTRE)
    dist = np.linalg.norm(r, axis=1)
    assert (dist >= _radius(body, r / dist[:, None]) * (1 - 1e-12)).all()


def test_features_are_layer_normalised_per_point():
    for gen in (DeviceSurface(3, 128, device="cpu", dtype=torch.float32),
                DeviceVolume(5, 128, device="cpu", dtype=torch.float32)):
        x = torch.empty((3000, 128), dtype=torch.float32)
        gen.fill(x)
        x = x.double().numpy()
        np.testing.assert_allclose(x.mean(axis=1), 0, atol=1e-5)
        np.testing.assert_allclose(x.var(axis=1), 1, atol=1e-3)


def test_gather_returns_the_mesh_rows_at_the_drawn_indices():
    """gather() generates each chunk that holds a drawn row as fill() does for
    the whole mesh and selects the drawn rows, bit for bit."""
    d = DeviceVolume(5, 64, device="cpu", dtype=torch.float32)
    # a 3,004,000-point mesh: chunks 0-2 full, chunk 3 holds 4,000 points
    source = 3 * G.CHUNK + 4000
    offs = np.array([3, 17, 250, 999, 3999])
    idx = np.concatenate([k * G.CHUNK + offs for k in (1, 3)])
    x = torch.empty((len(idx), 64), dtype=torch.float32)
    d.gather(x, idx, source)
    ref1 = d.features(d.points(1, G.CHUNK))[torch.from_numpy(offs)]
    ref3 = d.features(d.points(3, 4000))[torch.from_numpy(offs)]
    # fill() writes features(points(k, n_k)) at rows k*CHUNK.. of the mesh
    assert torch.equal(x[:5], ref1) and torch.equal(x[5:], ref3)


def test_training_subset_is_a_seeded_uniform_draw_without_replacement():
    from ts3_synth import WORKLOADS
    from ts3_synth.workloads import subset_indices
    wl = WORKLOADS["volume_2m_fp32"]
    idx = subset_indices(wl)
    assert len(idx) == wl.N == 2_000_000 and wl.source_N == 160_000_000
    assert (np.diff(idx) > 0).all() and idx[0] >= 0 and idx[-1] < wl.source_N
    assert np.array_equal(idx, subset_indices(wl))
    # uniform over the mesh: 160 equal bins, chi-square with 159 degrees of
    # freedom stays far below its 1e-6 tail (about 260)
    counts = np.bincount(idx * 160 // wl.source_N, minlength=160)
    chi2 = ((counts - wl.N / 160) ** 2 / (wl.N / 160)).sum()
    assert chi2 < 260, chi2
