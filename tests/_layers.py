"""Layer stand-ins for tests: same interface as moe_inputs.LayerInputs
(cfg, seed, bits, router, weight(), copy_headers(), slots_on())."""
import numpy as np

import moe_inputs as mi


def fp16_up(v: float) -> np.float16:
    h = np.float16(v)
    if float(h) < v:
        h = np.nextafter(h, np.float16(np.inf))
    return h


class GridLayer(mi.LayerInputs):
    """A layer whose expert weights lie exactly on the quantization grid of
    their expert's bit-width: every (row, group) is s*(q - z) with an fp16
    scale s, integer zero z, and both codes 0 and 2^b - 1 present, so
    quantization at that bit-width is lossless."""

    def weight(self, expert, kind):
        c = self.cfg
        R, K, g = c.rows(kind, expert), c.cols(kind, expert), c.group
        b = int(self.bits[expert])
        qmax = (1 << b) - 1
        r = mi.rng(self.seed, 77, 100 + 3 * expert + kind)
        G = K // g
        s = np.vectorize(fp16_up)(10.0 ** r.uniform(-3.6, -2.4, (R, G))).astype(np.float64)
        z = r.integers(0, qmax + 1, (R, G))
        q = r.integers(0, qmax + 1, (R, G, g))
        pos = np.argsort(r.random((R, G, g)), axis=2)[:, :, :2]
        np.put_along_axis(q, pos[:, :, :1], 0, axis=2)
        np.put_along_axis(q, pos[:, :, 1:], qmax, axis=2)
        w = s[:, :, None] * (q - z[:, :, None])
        return w.reshape(R, K).astype(np.float32)


class BitsOverride:
    """The same layer with every expert's bit-width replaced."""

    def __init__(self, layer, bits):
        self.cfg = layer.cfg
        self.seed = layer.seed
        self.router = layer.router
        self._layer = layer
        self.bits = np.full_like(layer.bits, bits) if np.isscalar(bits) else np.asarray(bits)

    def weight(self, e, kind):
        return self._layer.weight(e, kind)

    def copy_headers(self, kind):
        return self._layer.copy_headers(kind)

    def slots_on(self, kind, epoch=0):
        return self._layer.slots_on(kind, epoch)


class Pow2GridLayer(mi.LayerInputs):
    """Like GridLayer, but every scale is a power of two, so each weight
    s*(q - z) (|q - z| <= 255) is also exactly a binary16 value: quantizing the
    binary16 rounding of a row at its expert's bit-width is still lossless."""

    def weight(self, expert, kind):
        c = self.cfg
        R, K, g = c.rows(kind, expert), c.cols(kind, expert), c.group
        b = int(self.bits[expert])
        qmax = (1 << b) - 1
        r = mi.rng(self.seed, 78, 100 + 3 * expert + kind)
        G = K // g
        s = 2.0 ** r.integers(-12, -6, (R, G)).astype(np.float64)
        z = r.integers(0, qmax + 1, (R, G))
        q = r.integers(0, qmax + 1, (R, G, g))
        pos = np.argsort(r.random((R, G, g)), axis=2)[:, :, :2]
        np.put_along_axis(q, pos[:, :, :1], 0, axis=2)
        np.put_along_axis(q, pos[:, :, 1:], qmax, axis=2)
        w = s[:, :, None] * (q - z[:, :, None])
        return w.reshape(R, K).astype(np.float32)
