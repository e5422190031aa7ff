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
