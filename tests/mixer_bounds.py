"""Reference values and error bars for the mixer decode step when the GPU and
the oracle each carry their own float16 states from step to step (a test
helper: every reference value comes from the oracle).

Per step the float16 state S' = fp16(a S + c) is rounded on both sides from
different float32 / float64 values, and each side starts from its own
previous state.  With E the bound on |S_gpu - S_oracle| before the step:
  |S'_gpu - S'_oracle| <= a E + (both roundings: one float16 step of S',
  at most 2^-10 |S'| + 2^-24) + (float32 arithmetic in a S + c: well under
  2e-5 (|S'| + |S|)),
and a <= 1, so E grows by the last three terms per step.  The gated value
g = (S' C + D x) SiLU(z) then differs by at most |SiLU(z)| sum_n E |C_n|
plus float32 arithmetic (1e-5 of the magnitudes summed).
"""

import numpy as np

from oracle import mamba as MB

HEADDIM, D_STATE = 64, 128


def oracle_gate(z, conv, ssm, prm):
    """The oracle's step up to the gate for in_proj outputs z [B, Z]:
    (g [B, d_inner], new conv window, new SSM state (float16), C [B, N],
    SiLU(z) [B, d_inner], D x [B, d_inner])."""
    H = prm["A_log"].shape[0]
    di = H * HEADDIM
    zz, xBC, dt = MB.split_in_proj(z, di, D_STATE, H)
    u, conv_new = MB.conv_step(conv, xBC, prm["conv_w"], prm["conv_b"])
    x = u[:, :di].reshape(-1, H, HEADDIM)
    Bv, Cv = u[:, di:di + D_STATE], u[:, di + D_STATE:]
    y, ssm_new = MB.ssm_step(ssm, x, Bv, Cv, dt, prm["dt_bias"], prm["A_log"], prm["D"])
    sz = MB.silu(zz)
    dx = (np.asarray(prm["D"], np.float64)[None, :, None] * x).reshape(-1, di)
    return y.reshape(-1, di) * sz, conv_new, ssm_new, Cv, sz, dx


class StateBound:
    """Running bound E on |S_gpu - S_oracle| (elementwise, float64)."""

    def __init__(self, ssm0):
        self.prev = np.abs(np.asarray(ssm0, np.float16).astype(np.float64))
        self.E = np.zeros_like(self.prev)

    def step(self, ssm_new):
        a = np.abs(np.asarray(ssm_new, np.float16).astype(np.float64))
        self.E = self.E + 2.0 ** -10 * a + 2e-5 * (a + self.prev) + 2.0 ** -24
        self.prev = a
        return self.E

    def check(self, s_gpu, ssm_ref):
        d = np.abs(np.asarray(s_gpu, np.float16).astype(np.float64)
                   - np.asarray(ssm_ref, np.float16).astype(np.float64))
        bad = d > self.E * 1.001
        assert not bad.any(), f"SSM state: {int(bad.sum())} elements beyond the bound"

    def gate_bar(self, ssm_ref, C, sz, dx, g_ref):
        """Elementwise bar on |g_gpu - g_oracle| after `step`."""
        B = C.shape[0]
        E = self.E.reshape(B, -1, D_STATE)
        S = np.abs(np.asarray(ssm_ref, np.float16).astype(np.float64)).reshape(B, -1, D_STATE)
        Ca = np.abs(C)[:, None, :]
        prop = (E * Ca).sum(-1)                   # [B, d_inner]
        mag = (S * Ca).sum(-1) + np.abs(dx)
        return np.abs(sz) * (prop + 1e-5 * mag) + 1e-6 * np.abs(g_ref).max()
