"""Plain data carriers for a pinhole camera and the rasteriser constants.

The paper renders with 3D Gaussian Splatting and fixes none of its constants
(Method section); the defaults here are the readings this library uses, each a
runtime parameter of the C ABI.
"""
from dataclasses import dataclass, field

import numpy as np


@dataclass
class Camera:
    """World->camera pinhole: x_cam = R x_world + t, OpenCV axes (x right, y down,
    z forward); pixel (i, j) is sampled at (i + 0.5, j + 0.5)."""
    width: int
    height: int
    fx: float
    fy: float
    cx: float
    cy: float
    R: np.ndarray
    t: np.ndarray
    campos: np.ndarray
    near: float = 0.2

    @property
    def tiles(self):
        return ((self.width + 15) // 16, (self.height + 15) // 16)


@dataclass
class RasterParams:
    alpha_min: float = 1.0 / 255.0   # skip blends below this alpha
    alpha_max: float = 0.99          # clamp alpha to this
    t_min: float = 1e-4              # stop a pixel before transmittance falls below this
    eps2d: float = 0.3               # 2D covariance dilation, px^2
    radius_sigmas: float = 3.0       # support radius in sigmas of the major axis
    guard: float = 1.3               # guard band on the view frustum used in the Jacobian
    sh_degree: int = 0
    fb_stop: bool = False            # compositing-aware stop: (1 - F_alpha) T < t_min ends a pixel


def look_at(campos, target, width, height, fov_x_deg=60.0, up=(0.0, 0.0, 1.0), near=0.2):
    """Pinhole camera at campos looking at target, focal length from the
    horizontal field of view, principal point at the image centre."""
    campos = np.asarray(campos, np.float64)
    fwd = np.asarray(target, np.float64) - campos
    fwd /= np.linalg.norm(fwd)
    right = np.cross(fwd, np.asarray(up, np.float64))
    right /= np.linalg.norm(right)
    down = np.cross(fwd, right)
    R = np.stack([right, down, fwd]).astype(np.float32)
    t = (-(R.astype(np.float64) @ campos)).astype(np.float32)
    # every field is stored in fp32, as the C structures hold it
    f = float(np.float32(width / (2.0 * np.tan(np.deg2rad(fov_x_deg) / 2.0))))
    return Camera(width=width, height=height, fx=f, fy=f, cx=width / 2.0, cy=height / 2.0,
                  R=R, t=t, campos=campos.astype(np.float32), near=float(np.float32(near)))
