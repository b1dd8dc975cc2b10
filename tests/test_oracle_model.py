"""The denoising-step oracle against its pins, and planted mistakes in it (on
the CPU) that at least one pin must catch."""
import numpy as np
import pytest

from oracle import dit_model as M
from oracle_model_pins import ALL_CHECKS


@pytest.mark.parametrize("check", ALL_CHECKS, ids=[c.__name__ for c in ALL_CHECKS])
def test_pin(check):
    check()


orig = {n: getattr(M, n) for n in dir(M) if callable(getattr(M, n))}


def m_patch_token_hw(lat, patch):
    """tokens in (f, w, h) order"""
    C, FL, HL, WL = lat.shape
    pt, ph, pw = patch
    v = lat.reshape(C, FL // pt, pt, HL // ph, ph, WL // pw, pw).transpose(1, 5, 3, 0, 2, 4, 6)
    return v.reshape(-1, C * pt * ph * pw)


def m_patch_channel_last(lat, patch):
    """patch vector in (i, j, k, c) order"""
    C, FL, HL, WL = lat.shape
    pt, ph, pw = patch
    v = lat.reshape(C, FL // pt, pt, HL // ph, ph, WL // pw, pw).transpose(1, 3, 5, 2, 4, 6, 0)
    return v.reshape(-1, C * pt * ph * pw)


def m_unpatch_jk(tok, C, grid, patch):
    """unpatchify with the in-patch height and width offsets swapped"""
    F_, H, W = grid
    pt, ph, pw = patch
    v = tok.reshape(F_, H, W, C, pt, ph, pw).transpose(3, 0, 4, 1, 6, 2, 5)
    return v.reshape(C, F_ * pt, H * pw, W * ph) if ph == pw else v.reshape(-1)


def m_final_shift_scale(x, c, req, eps, mw):
    D = x.shape[1]
    w = dict(mw, w_hmod=np.concatenate([mw["w_hmod"][D:], mw["w_hmod"][:D]]),
             b_hmod=np.concatenate([mw["b_hmod"][D:], mw["b_hmod"][:D]]))
    return orig["final_layer"](x, c, req, eps, w)


def m_final_no_silu(x, c, req, eps, mw):
    import oracle.dit_block as O
    m = O.linear(c, mw["w_hmod"], mw["b_hmod"])
    D = x.shape[1]
    h = O.modulate(O.layer_norm(x, eps), m[:, :D][req], m[:, D:][req])
    return O.linear(h, mw["w_out"], mw["b_out"])


def m_final_no_bias(x, c, req, eps, mw):
    return orig["final_layer"](x, c, req, eps, mw) - mw["b_out"]


def m_euler_sign(latent, v, dt):
    return latent - dt * v


def m_euler_half(latent, v, dt):
    return latent + 0.5 * dt * v


def m_shared_time_silu(t, freq_dim, mw):
    import oracle.dit_block as O
    return O.silu(orig["shared_time"](t, freq_dim, mw))


def m_shared_time_no_b2(t, freq_dim, mw):
    return orig["shared_time"](t, freq_dim, mw) - mw["b_t2"]


MUTANTS = {
    "patchify": [m_patch_token_hw, m_patch_channel_last],
    "unpatchify": [m_unpatch_jk],
    "final_layer": [m_final_shift_scale, m_final_no_silu, m_final_no_bias],
    "euler_step": [m_euler_sign, m_euler_half],
    "shared_time": [m_shared_time_silu, m_shared_time_no_b2],
}
CASES = [(name, m) for name, ms in MUTANTS.items() for m in ms]


@pytest.mark.parametrize("name,mutant", CASES, ids=[m.__name__ for _, m in CASES])
def test_mutant_caught(monkeypatch, name, mutant):
    monkeypatch.setattr(M, name, mutant)
    failed = []
    for c in ALL_CHECKS:
        try:
            c()
        except (AssertionError, ValueError):
            failed.append(c.__name__)
    assert failed, f"no pin catches {mutant.__name__} ({mutant.__doc__ or ''})"


def test_dt_per_request_order(monkeypatch):
    """dt given to the wrong request (reversed) is caught."""
    real = M.denoise_step

    def swapped(cfg, vl, C, patch, latent, t, dt, *a, **k):
        return real(cfg, vl, C, patch, latent, t, np.asarray(dt)[::-1].copy(), *a, **k)

    monkeypatch.setattr(M, "denoise_step", swapped)
    import oracle_model_pins as P
    with pytest.raises(AssertionError):
        P.check_step_requests_independent()
