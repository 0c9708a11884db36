"""The C ABI on the host: the library loads, exports what include/sao.h declares,
and rejects invalid arguments synchronously before any device work.

No call here reaches a kernel launch: every case fails validation or is the
T == 0 no-op, so the pointers passed are never dereferenced.
"""
import os
import re

import pytest

from paper_2607_07508_amd import binding

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "sao.h")

OK, ERR_NULL, ERR_SHAPE, ERR_VALUE, ERR_DTYPE, ERR_WORKSPACE = 0, 1, 2, 3, 4, 5
FAKE = 0x10000          # 16- and 256-byte aligned, never dereferenced
FAKE_ODD = 0x10008      # 8 mod 16


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"\b(sao_[a-z_0-9]+)\s*\(", text)))


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(binding.LIB_PATH):
        pytest.skip("libsao.so not built")
    return binding.lib()


def test_exports_every_declared_symbol(L):
    names = declared_functions()
    assert set(names) >= {"sao_token_logprob", "sao_advantage", "sao_clipped_loss", "sao_loss_backward"}
    for n in names:
        assert hasattr(L, n), n
    assert set(names) == set(binding.EXPORTS)


def test_version_and_strings(L):
    assert L.sao_version().decode().count(".") == 2
    for code in range(7):
        assert L.sao_status_string(code)


def logprob(L, hidden=FAKE, ldh=64, w=FAKE, ldw=64, tgt=FAKE, mask=None, T=16, H=64, V=1000, dt=0,
            logp=FAKE, lse=FAKE, ws=FAKE, ws_bytes=1 << 40):
    return L.sao_token_logprob(hidden, ldh, w, ldw, tgt, mask, T, H, V, dt, logp, lse, None, ws, ws_bytes, None)


def test_logprob_validation(L):
    assert logprob(L, hidden=None) == ERR_NULL
    assert logprob(L, lse=None) == ERR_NULL
    assert logprob(L, T=-1) == ERR_SHAPE
    assert logprob(L, H=12, ldh=16, ldw=16) == ERR_SHAPE            # H not a multiple of 8
    assert logprob(L, V=0) == ERR_SHAPE
    assert logprob(L, ldh=32) == ERR_SHAPE                          # ld < H
    assert logprob(L, ldw=68) == ERR_SHAPE                          # ld not a multiple of 8
    assert logprob(L, hidden=FAKE_ODD) == ERR_SHAPE                 # misaligned
    assert logprob(L, dt=7) == ERR_DTYPE
    assert logprob(L, ws_bytes=16) == ERR_WORKSPACE
    assert logprob(L, ws=None) == ERR_NULL
    assert logprob(L, ws=FAKE + 16) == ERR_WORKSPACE               # not 256-byte aligned
    assert logprob(L, T=0) == OK                                    # no-op
    # row strides: the tile engine's 32-bit lane offsets allow 2^24 bytes per row
    assert logprob(L, ldh=(1 << 23) + 8) == ERR_SHAPE                # bf16
    assert logprob(L, ldw=(1 << 23) + 8) == ERR_SHAPE
    assert logprob(L, ldw=1 << 23, ws_bytes=16) == ERR_WORKSPACE     # the largest stride passes the shape checks
    assert logprob(L, ldh=(1 << 22) + 8, dt=1) == ERR_SHAPE          # fp32
    assert logprob(L, ldh=1 << 22, dt=1, ws_bytes=16) == ERR_WORKSPACE
    assert b"workspace" in L.sao_last_error_message() or L.sao_last_error_message() == b""


def test_advantage_validation(L):
    def adv(vals=FAKE, B=2, T=10, gamma=1.0, lam=1.0, alpha=0.0, adv_out=FAKE, ws=FAKE, ws_bytes=256):
        return L.sao_advantage(vals, FAKE, FAKE, FAKE, B, T, gamma, lam, alpha, adv_out, FAKE, None, None,
                               ws, ws_bytes, None)
    assert adv(vals=None) == ERR_NULL
    assert adv(adv_out=None) == ERR_NULL
    assert adv(B=0) == ERR_SHAPE
    assert adv(T=-3) == ERR_SHAPE
    assert adv(gamma=1.5) == ERR_VALUE
    assert adv(gamma=float("nan")) == ERR_VALUE
    assert adv(lam=-0.1) == ERR_VALUE
    assert adv(alpha=float("inf")) == ERR_VALUE
    assert adv(alpha=-1.5) == ERR_VALUE                               # alpha == 0 selects the fixed lambda
    assert adv(alpha=0.0, ws_bytes=4) == ERR_WORKSPACE
    assert adv(ws=None) == ERR_NULL
    assert adv(ws_bytes=4) == ERR_WORKSPACE
    assert adv(T=0) == OK


def test_step_advantage_validation(L):
    def st(vals=FAKE, B=2, T=10, gamma=1.0, lam=1.0, alpha=0.0, form=0, ws=FAKE, ws_bytes=1 << 20):
        return L.sao_step_advantage(vals, FAKE, FAKE, FAKE, B, T, gamma, lam, alpha, form, FAKE, FAKE, None, None,
                                    None, ws, ws_bytes, None)
    assert st(vals=None) == ERR_NULL
    assert st(B=0) == ERR_SHAPE
    assert st(T=-1) == ERR_SHAPE
    assert st(gamma=-0.5) == ERR_VALUE
    assert st(lam=2.0) == ERR_VALUE
    assert st(alpha=float("nan")) == ERR_VALUE
    assert st(alpha=-0.5) == ERR_VALUE
    assert st(form=2) == ERR_VALUE
    assert st(ws=None) == ERR_NULL
    assert st(ws_bytes=64) == ERR_WORKSPACE
    assert st(T=0) == OK
    assert binding.workspace_size(binding.OP_STEP_ADVANTAGE, 1000, 1, 1, 1) >= 24 * 1000


def test_baseline_validation(L):
    def grp(adv=FAKE, B=8, T=100, G=4, eps=1e-6, tr=FAKE, ws=FAKE, ws_bytes=256):
        return L.sao_group_advantage(FAKE, FAKE, FAKE, B, T, G, eps, adv, tr, FAKE, None, None, ws, ws_bytes, None)
    assert grp(adv=None) == ERR_NULL
    assert grp(tr=None) == ERR_NULL
    assert grp(G=3) == ERR_SHAPE                 # B not a multiple of the group size
    assert grp(G=0) == ERR_SHAPE
    assert grp(eps=-1.0) == ERR_VALUE
    assert grp(eps=float("inf")) == ERR_VALUE
    assert grp(ws_bytes=0) == ERR_WORKSPACE
    assert grp(T=0) == OK

    def rm(hist=FAKE, seen=FAKE, n_keys=2, window=8, B=4, T=100, ws=FAKE, ws_bytes=256):
        return L.sao_running_mean_advantage(FAKE, FAKE, FAKE, B, T, None, n_keys, window, hist, seen, FAKE, FAKE,
                                            FAKE, None, None, ws, ws_bytes, None)
    assert rm(hist=None) == ERR_NULL
    assert rm(seen=None) == ERR_NULL
    assert rm(n_keys=0) == ERR_SHAPE
    assert rm(window=0) == ERR_SHAPE
    assert rm(B=0) == ERR_SHAPE
    assert rm(ws=None) == ERR_NULL
    assert rm(T=0) == OK


def test_loss_validation(L):
    def loss(T=10, el=0.2, eh=0.2, g=FAKE, ws=FAKE, ws_bytes=1 << 30):
        return L.sao_clipped_loss(FAKE, FAKE, FAKE, FAKE, T, el, eh, None, FAKE, g, FAKE, FAKE, ws, ws_bytes,
                                  None)
    assert loss(g=None) == ERR_NULL
    assert loss(el=-0.1) == ERR_VALUE
    assert loss(eh=float("inf")) == ERR_VALUE
    assert loss(eh=float("nan")) == ERR_VALUE
    assert loss(ws_bytes=8) == ERR_WORKSPACE
    assert loss(T=0) == OK


def test_loss_noalloc_validation(L):
    def loss(T=10, el=0.2, eh=0.2, g=FAKE, lp=FAKE):
        return L.sao_clipped_loss_noalloc(lp, FAKE, FAKE, FAKE, T, el, eh, None, FAKE, g, FAKE, FAKE, None)
    assert loss(g=None) == ERR_NULL
    assert loss(lp=None) == ERR_NULL
    assert loss(T=-1) == ERR_SHAPE
    assert loss(el=-0.1) == ERR_VALUE
    assert loss(eh=float("nan")) == ERR_VALUE
    assert loss(T=0) == OK


def test_ppo_loss_validation(L):
    def ppo(lold=FAKE, behav=None, T=10, el=0.2, eh=0.28, counts=FAKE, ws=FAKE, ws_bytes=1 << 30):
        return L.sao_ppo_loss(FAKE, lold, behav, FAKE, FAKE, T, el, eh, None, FAKE, FAKE, FAKE, counts, ws,
                              ws_bytes, None)
    assert ppo(lold=None) == ERR_NULL
    assert ppo(counts=None) == ERR_NULL
    assert ppo(T=-1) == ERR_SHAPE
    assert ppo(el=float("nan")) == ERR_VALUE
    assert ppo(eh=-1.0) == ERR_VALUE
    assert ppo(ws=None) == ERR_NULL
    assert ppo(ws_bytes=8) == ERR_WORKSPACE
    assert ppo(T=0) == OK
    assert ppo(T=0, behav=FAKE) == OK


def test_explained_variance_validation(L):
    def ev(values=FAKE, moments=FAKE, out=FAKE, T=10, ws=FAKE, ws_bytes=1 << 20):
        return L.sao_explained_variance(values, FAKE, FAKE, T, moments, out, ws, ws_bytes, None)
    assert ev(values=None) == ERR_NULL
    assert ev(moments=None) == ERR_NULL
    assert ev(T=-5) == ERR_SHAPE
    assert ev(ws=None) == ERR_NULL
    assert ev(ws_bytes=8) == ERR_WORKSPACE
    assert ev(ws=FAKE + 8) == ERR_WORKSPACE
    assert ev(T=0, out=None) == OK


def test_backward_validation(L):
    def bwd(dh=FAKE, dw=FAKE, T=16, H=64, V=100, dt=0, ws_bytes=1 << 40):
        return L.sao_loss_backward(FAKE, H, FAKE, H, FAKE, FAKE, FAKE, T, H, V, dt, dh, dw, FAKE, ws_bytes,
                                   None)
    assert bwd(dh=None) == ERR_NULL
    assert bwd(dw=FAKE_ODD) == ERR_SHAPE
    assert bwd(H=0) == ERR_SHAPE
    assert bwd(dt=2) == ERR_DTYPE
    assert bwd(ws_bytes=100) == ERR_WORKSPACE
    assert L.sao_loss_backward(FAKE, 64, FAKE, (1 << 23) + 8, FAKE, FAKE, FAKE, 16, 64, 100, 0, FAKE, FAKE, FAKE,
                               1 << 40, None) == ERR_SHAPE
    assert bwd(T=0) == OK


def test_value_validation(L):
    def fwd(hidden=FAKE, w=FAKE, v=FAKE, T=16, H=64, ld=64, dt=0):
        return L.sao_value_forward(hidden, ld, w, T, H, dt, v, None, 0, None)
    assert fwd(hidden=None) == ERR_NULL
    assert fwd(v=None) == ERR_NULL
    assert fwd(H=12, ld=16) == ERR_SHAPE
    assert fwd(ld=32) == ERR_SHAPE
    assert fwd(w=FAKE_ODD) == ERR_SHAPE
    assert fwd(dt=5) == ERR_DTYPE
    assert fwd(T=-2) == ERR_SHAPE
    assert fwd(T=0) == OK

    def vl(dh=FAKE, ret=FAKE, T=16, H=64, ws=FAKE, ws_bytes=1 << 30, dt=0):
        return L.sao_value_loss(FAKE, H, FAKE, FAKE, ret, FAKE, T, H, None, dt, FAKE, dh, FAKE, ws, ws_bytes, None)
    assert vl(ret=None) == ERR_NULL
    assert vl(dh=None) == ERR_NULL
    assert vl(dh=FAKE_ODD) == ERR_SHAPE
    assert vl(H=0) == ERR_SHAPE
    assert vl(dt=3) == ERR_DTYPE
    assert vl(ws_bytes=8) == ERR_WORKSPACE
    assert vl(ws=None) == ERR_NULL
    assert vl(T=0) == OK


def test_workspace_sizes(L):
    ws = binding.workspace_size
    assert ws(binding.OP_ADVANTAGE, 1000, 1, 1, 0) == 768     # segments flag + 64 count slots
    assert ws(binding.OP_LOGPROB, 0, 2048, 151936, 0) == 0
    assert ws(binding.OP_LOGPROB, -1, 2048, 151936, 0) == 0
    small = ws(binding.OP_LOGPROB, 1000, 64, 1000, 1)
    assert small > 1000 * 64 * 4
    # the backward dz scratch is one vocabulary block (in two layouts), not T x V
    big = ws(binding.OP_BACKWARD, 65536, 2048, 151936, 0)
    assert big < 65536 * 151936 * 2 // 2
    assert ws(binding.OP_LOSS, 1 << 26, 1, 1, 1) < 1 << 20
    assert ws(binding.OP_PPO_LOSS, 12345, 1, 1, 1) == ws(binding.OP_LOSS, 12345, 1, 1, 1)
    assert 0 < ws(binding.OP_EXPLAINED_VARIANCE, 1 << 26, 1, 1, 1) < 1 << 20
    # value loss: per-128-row partials of dw_v, far below the hidden states themselves
    assert 0 < ws(binding.OP_VALUE, 32768, 6144, 1, 0) < 32768 * 6144 * 2 // 16


def _block_rule(T, H, V, esize):
    """The backward's vocabulary block as include/sao.h states it for
    sao_workspace_size."""
    from math import gcd
    tiles_t = -(-T // 256)
    vt = 32768
    while vt < 65536 and tiles_t * (vt // 256) < 8192:
        vt *= 2
    n = -(-V // vt)
    b = -(-(-(-V // n)) // 256)
    m = 256 // gcd(256, -(-H // 256))
    if n > 1:
        up = -(-b // m) * m
        if up <= vt // 256 and 256 * up * H * esize <= 256 << 20:
            b = up
        elif b >= m:
            b = b // m * m
    return 256 * b


@pytest.mark.parametrize("T,H,V,dt", [
    (65536, 2048, 151936, 0),   # rounded up to whole dW rounds: 4 x 32768 + 20864
    (65536, 2048, 151936, 1),   # fp32: 256 x 128 x 2048 x 4 bytes is exactly 256 MiB, still rounded up
    (65536, 4096, 151936, 1),   # fp32 at H = 4096: 32768-row blocks would not fit, rounded down to 28672
    (32768, 6144, 151552, 0),   # W's block beyond the cache: rounded down to 24576
    (8192, 2048, 151936, 0),    # a short chunk: 65536-row target, 2 x 57344 + 37248
    (640, 64, 140000, 0),       # H = 64: 256-tile multiples
    (65536, 2048, 20000, 0),    # a single block: V rounded to a whole tile
    (3000, 768, 99999, 1),      # H = 768: a multiple of 256 tiles, the whole 65536-row target
    (65536, 2304, 151936, 0),   # H = 2304: 256-tile multiples exceed the target, blocks left equal
])
def test_backward_block_rule(L, T, H, V, dt):
    # the workspace differs between two vocabularies by the dz block alone
    # (esize x round_up(T, 256) x Vb bytes); V = 256 gives a one-tile block
    ws = binding.workspace_size
    esize = 2 if dt == 0 else 4
    t_pad = -(-T // 256) * 256
    d = ws(binding.OP_BACKWARD, T, H, V, dt) - ws(binding.OP_BACKWARD, T, H, 256, dt)
    assert d % (esize * t_pad) == 0
    assert d // (esize * t_pad) + 256 == _block_rule(T, H, V, esize)


def test_error_message_is_per_thread(L):
    # Two threads fail with different errors at the same time; each reads its own
    # message (the library keeps the last message per calling thread).
    import threading
    barrier = threading.Barrier(2)
    seen = {}

    def null_case():
        for _ in range(200):
            barrier.wait()
            code = L.sao_clipped_loss(None, FAKE, FAKE, FAKE, 16, 0.2, 0.2, None, FAKE, FAKE, FAKE, FAKE,
                                      None, 0, None)
            barrier.wait()
            seen.setdefault("null", set()).add((code, L.sao_last_error_message()))

    def value_case():
        for _ in range(200):
            barrier.wait()
            code = L.sao_clipped_loss(FAKE, FAKE, FAKE, FAKE, 16, -1.0, 0.2, None, FAKE, FAKE, FAKE, FAKE,
                                      None, 0, None)
            barrier.wait()
            seen.setdefault("value", set()).add((code, L.sao_last_error_message()))

    threads = [threading.Thread(target=null_case), threading.Thread(target=value_case)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert len(seen["null"]) == 1 and len(seen["value"]) == 1
    (code_n, msg_n), = seen["null"]
    (code_v, msg_v), = seen["value"]
    assert code_n == ERR_NULL and b"required" in msg_n
    assert code_v == ERR_VALUE and b"eps" in msg_v
