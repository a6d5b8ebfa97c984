"""Host-side checks of the C ABI: the library loads, exports every function
that include/dqn.h declares, reports the documented layout, and rejects bad
arguments with the documented status before enqueueing anything.  No kernel
is launched here; these run without a GPU."""
import ctypes
import os
import re

import pytest

import dqn_inputs as di
import paper_1508_04186_amd as dq
from paper_1508_04186_amd import native

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def header_functions(names=None):
    inc = os.path.join(ROOT, "include")
    names = names or sorted(f for f in os.listdir(inc) if f.endswith(".h"))
    txt = "".join(open(os.path.join(inc, f)).read() for f in names)
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"^\s*(?:const\s+)?\w+\**\s+\**(\w+)\s*\(", txt, flags=re.M)))


def test_header_declares_the_four_calls():
    fns = header_functions(["dqn.h"])
    for f in ("replay_gather", "dqn_forward", "dqn_forward_replay", "dqn_td_gradient", "dqn_td_gradient_replay",
              "ps_apply_update", "dqn_param_count", "dqn_param_offset", "dqn_workspace_bytes", "dqn_status_string"):
        assert f in fns


def test_library_exports_every_declared_symbol():
    L = dq.lib()
    for f in header_functions():
        assert hasattr(L, f), f
    # extern "C": no mangled names needed
    assert isinstance(ctypes.cast(L.dqn_forward, ctypes.c_void_p).value, int)


@pytest.mark.parametrize("net,shape", [(dq.NET_SMALL, di.NET_S), (dq.NET_LARGE, di.NET_L)])
def test_param_layout_matches_documentation(net, shape):
    assert dq.dqn_param_count(net) == shape.param_count()
    sl = shape.slices()
    L = len(net.conv)
    for l in range(L):
        assert dq.dqn_param_offset(net, l, False) == sl[f"conv{l+1}.W"][0]
        assert dq.dqn_param_offset(net, l, True) == sl[f"conv{l+1}.b"][0]
    assert dq.dqn_param_offset(net, L, False) == sl["fc1.W"][0]
    assert dq.dqn_param_offset(net, L, True) == sl["fc1.b"][0]
    assert dq.dqn_param_offset(net, L + 1, False) == sl["fc2.W"][0]
    assert dq.dqn_param_offset(net, L + 1, True) == sl["fc2.b"][0]
    with pytest.raises(dq.DqnError) as e:
        dq.dqn_param_offset(net, L + 2, False)
    assert e.value.status == dq.DQN_EINVAL


def test_documented_offsets_small_net():
    assert [dq.dqn_param_offset(dq.NET_SMALL, l, b) for l in range(4) for b in (0, 1)] == \
        [0, 4096, 4112, 12304, 12336, 675888, 676144, 677680]
    assert dq.dqn_param_count(dq.NET_SMALL) == 677686
    assert dq.dqn_param_count(dq.NET_LARGE) == 1693362


def test_unsupported_networks_and_bad_batch():
    bad = dq.Net(4, 84, 84, ((16, 8, 4), (32, 4, 2)), 256, 7)
    with pytest.raises(dq.DqnError) as e:
        dq.dqn_param_count(bad)
    assert e.value.status == dq.DQN_EUNSUPPORTED
    with pytest.raises(dq.DqnError) as e:
        dq.dqn_workspace_bytes(dq.NET_SMALL, 0, dq.DQN_OP_TD_GRADIENT)
    assert e.value.status == dq.DQN_EINVAL
    with pytest.raises(dq.DqnError):
        dq.dqn_workspace_bytes(dq.NET_SMALL, 4, 7)
    fp16 = dq.Net(4, 84, 84, ((16, 8, 4), (32, 4, 2)), 256, 6, precision=3)
    with pytest.raises(dq.DqnError) as e:
        dq.dqn_param_count(fp16)
    assert e.value.status == dq.DQN_EUNSUPPORTED


def test_bf16_variant_is_large_network_only():
    assert dq.dqn_param_count(dq.NET_LARGE_BF16) == dq.dqn_param_count(dq.NET_LARGE)
    for l in range(5):
        for b in (0, 1):
            assert dq.dqn_param_offset(dq.NET_LARGE_BF16, l, b) == dq.dqn_param_offset(dq.NET_LARGE, l, b)
    small_bf16 = dq.Net(4, 84, 84, ((16, 8, 4), (32, 4, 2)), 256, 6, precision=dq.DQN_BF16)
    with pytest.raises(dq.DqnError) as e:
        dq.dqn_workspace_bytes(small_bf16, 32, dq.DQN_OP_TD_GRADIENT)
    assert e.value.status == dq.DQN_EUNSUPPORTED


def test_workspace_grows_with_batch():
    for net in (dq.NET_SMALL, dq.NET_LARGE, dq.NET_LARGE_BF16):
        for op in (dq.DQN_OP_FORWARD, dq.DQN_OP_TD_GRADIENT):
            a = dq.dqn_workspace_bytes(net, 32, op)
            b = dq.dqn_workspace_bytes(net, 2048, op)
            assert 0 < a < b and a % 256 == 0 and b % 256 == 0


# Raw C calls with fake (never dereferenced) device addresses: every one of
# these must fail the host checks, so nothing is launched.  They run only
# where no GPU is visible, so a missing check can never become a launch on
# bogus pointers.
FAKE = 0x7F0000000000


def _no_gpu():
    try:
        import torch
        return not torch.cuda.is_available()
    except Exception:
        return True


fake_ptr_test = pytest.mark.skipif(not _no_gpu(), reason="fake-pointer checks run only without a GPU")


def _cnet(net):
    return ctypes.byref(native._cnet(net))


@fake_ptr_test
def test_td_gradient_argument_errors():
    L = dq.lib()
    n = dq.NET_SMALL
    P = dq.dqn_param_count(n)
    ws = dq.dqn_workspace_bytes(n, 8, dq.DQN_OP_TD_GRADIENT)
    args = dict(theta=FAKE, tt=FAKE, s=FAKE + 2**30, sn=FAKE + 2**31, a=FAKE, r=FAKE, t=FAKE, B=8,
                g=FAKE + 2**33, loss=FAKE, q=None, y=None, ws=FAKE + 2**34, wsb=ws)

    def call(**kw):
        a = dict(args, **kw)
        return L.dqn_td_gradient(_cnet(n), a["theta"], a["tt"], a["s"], a["sn"], a["a"], a["r"],
                                 a["t"], a["B"], ctypes.c_float(0.99), a["g"], a["loss"], a["q"],
                                 a["y"], a["ws"], a["wsb"], None)
    assert call(theta=None) == dq.DQN_EINVAL
    assert call(s=None) == dq.DQN_EINVAL
    assert call(g=None) == dq.DQN_EINVAL
    assert call(B=0) == dq.DQN_EINVAL
    assert call(B=-3) == dq.DQN_EINVAL
    assert call(wsb=ws - 1) == dq.DQN_EWORKSPACE
    assert call(ws=FAKE + 2**34 + 8) == dq.DQN_EINVAL            # misaligned workspace
    assert call(g=FAKE + 4 * (P // 2)) == dq.DQN_EINVAL           # grad overlaps theta
    assert call(g=FAKE, tt=FAKE + 2**33) == dq.DQN_EINVAL         # grad overlaps theta_target
    bad = dq.Net(4, 84, 84, ((16, 8, 4),), 256, 6)
    assert L.dqn_td_gradient(_cnet(bad), FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 8,
                             ctypes.c_float(0.99), FAKE + 2**33, FAKE, None, None, FAKE, ws,
                             None) == dq.DQN_EUNSUPPORTED


@fake_ptr_test
def test_forward_argument_errors():
    L = dq.lib()
    n = dq.NET_LARGE
    ws = dq.dqn_workspace_bytes(n, 16, dq.DQN_OP_FORWARD)

    def call(eps=0.0, draws=None, B=16, wsb=ws, theta=FAKE):
        return L.dqn_forward(_cnet(n), theta, FAKE, B, ctypes.c_float(eps), draws, FAKE, FAKE,
                             FAKE + 2**34, wsb, None)
    assert call(eps=0.05, draws=None) == dq.DQN_EINVAL   # exploration needs draws
    assert call(eps=-0.1, draws=FAKE) == dq.DQN_EINVAL
    assert call(eps=1.5, draws=FAKE) == dq.DQN_EINVAL
    assert call(eps=float("nan"), draws=FAKE) == dq.DQN_EINVAL
    assert call(B=0) == dq.DQN_EINVAL
    assert call(wsb=ws - 256) == dq.DQN_EWORKSPACE
    assert call(theta=None) == dq.DQN_EINVAL


@fake_ptr_test
def test_gather_argument_errors():
    L = dq.lib()
    rp = native._CReplay()
    rp.frames, rp.action, rp.reward, rp.terminal = FAKE, FAKE, FAKE, FAKE
    rp.record_stride, rp.size, rp.c, rp.h, rp.w = 28224, 100, 4, 84, 84

    def call(B=4, s=FAKE + 2**30, sn=FAKE + 2**31, **kw):
        for k, v in kw.items():
            setattr(rp, k, v)
        return L.replay_gather(ctypes.byref(rp), FAKE, B, s, sn, None, None, None, None)
    assert call(s=None) == dq.DQN_EINVAL
    assert call(B=0) == dq.DQN_EINVAL
    assert call(s=FAKE + 2**30 + 4) == dq.DQN_EINVAL          # misaligned output
    assert call(record_stride=28224 + 8) == dq.DQN_EINVAL     # stride not a multiple of 16
    assert call(record_stride=1000) == dq.DQN_EINVAL          # stride below record size
    rp.record_stride = 28224
    assert call(size=1) == dq.DQN_EINVAL                      # needs two records for s'
    rp.size = 100
    assert call(h=83, w=83) == dq.DQN_EINVAL                  # record not a multiple of 16 bytes


@fake_ptr_test
def test_validate_argument_errors():
    L = dq.lib()
    rp = native._CReplay()
    rp.frames, rp.action, rp.reward, rp.terminal = FAKE, FAKE, FAKE, FAKE
    rp.record_stride, rp.size, rp.c, rp.h, rp.w = 28224, 100, 4, 84, 84
    assert L.replay_gather_validate(None, FAKE, 4, 1, FAKE + 64, None) == dq.DQN_EINVAL
    assert L.replay_gather_validate(ctypes.byref(rp), None, 4, 1, FAKE + 64, None) == dq.DQN_EINVAL
    assert L.replay_gather_validate(ctypes.byref(rp), FAKE, 0, 1, FAKE + 64, None) == dq.DQN_EINVAL
    assert L.replay_gather_validate(ctypes.byref(rp), FAKE, 4, 1, None, None) == dq.DQN_EINVAL
    rp.size = 1                                               # no transition has a next state
    assert L.replay_gather_validate(ctypes.byref(rp), FAKE, 4, 1, FAKE + 64, None) == dq.DQN_EINVAL


@fake_ptr_test
def test_fill_argument_errors():
    L = dq.lib()
    rp = native._CReplay()
    rp.frames, rp.action, rp.reward, rp.terminal = FAKE, FAKE, FAKE, FAKE
    rp.record_stride, rp.size, rp.c, rp.h, rp.w = 28224, 100, 4, 84, 84

    def call(n_actions=6, **kw):
        for k, v in kw.items():
            setattr(rp, k, v)
        return L.replay_fill_synthetic(ctypes.byref(rp), n_actions, 7, None)
    assert call(n_actions=0) == dq.DQN_EINVAL
    assert call(n_actions=257) == dq.DQN_EINVAL
    assert call(frames=FAKE + 4) == dq.DQN_EINVAL             # frames not 16-byte aligned
    rp.frames = FAKE
    assert call(record_stride=28224 + 8) == dq.DQN_EINVAL     # stride not a multiple of 16
    assert call(record_stride=28224 - 16) == dq.DQN_EINVAL    # stride below c frames
    rp.record_stride = 28224
    assert call(size=0) == dq.DQN_EINVAL
    rp.size = 100
    assert call(h=80, w=80) == dq.DQN_EINVAL                  # the stream's frames are 84 x 84
    rp.h, rp.w = 84, 84
    assert call(c=0) == dq.DQN_EINVAL
    rp.c = 4
    assert call(terminal=None) == dq.DQN_EINVAL


@fake_ptr_test
def test_apply_argument_errors():
    L = dq.lib()

    def call(rule=0, th=FAKE, out=FAKE, st=None, g=FAKE + 2**32, n=1000, lr=0.1):
        return L.ps_apply_update(rule, th, out, st, g, n, ctypes.c_float(lr), ctypes.c_float(0.9),
                                 ctypes.c_float(0.0), None)
    assert call(rule=5) == dq.DQN_EINVAL
    assert call(rule=1, st=None) == dq.DQN_EINVAL            # RMSProp needs its state
    assert call(rule=2, st=None) == dq.DQN_EINVAL
    assert call(n=0) == dq.DQN_EINVAL
    assert call(g=FAKE + 64) == dq.DQN_EINVAL                # grad overlaps theta_out
    assert call(out=FAKE + 64) == dq.DQN_EINVAL              # partial overlap of in and out
    assert call(rule=2, st=FAKE + 2**32 + 16) == dq.DQN_EINVAL  # state overlaps grad
    assert call(th=FAKE + 2) == dq.DQN_EINVAL                # misaligned
    assert call(lr=float("inf")) == dq.DQN_EINVAL


@fake_ptr_test
def test_peak_check_argument_errors():
    L = dq.lib()
    assert L.dqn_profile_mfma_peak(7, 16, 16, FAKE, None) == dq.DQN_EINVAL       # unknown dtype
    assert L.dqn_profile_mfma_peak(0, 0, 16, FAKE, None) == dq.DQN_EINVAL
    assert L.dqn_profile_mfma_peak(1, 16, 0, FAKE, None) == dq.DQN_EINVAL
    assert L.dqn_profile_mfma_peak(0, 16, 16, None, None) == dq.DQN_EINVAL
    assert L.dqn_profile_stream_copy(FAKE, FAKE + 4096, 100, 8, None) == dq.DQN_EINVAL   # not whole vectors
    assert L.dqn_profile_stream_copy(FAKE, FAKE + 64, 4096, 8, None) == dq.DQN_EINVAL    # overlap
    assert L.dqn_profile_stream_copy(FAKE + 4, FAKE + 8192, 4096, 8, None) == dq.DQN_EINVAL  # misaligned
    assert L.dqn_profile_stream_copy(FAKE, FAKE + 8192, 4096, 0, None) == dq.DQN_EINVAL


@fake_ptr_test
def test_actor_argument_errors():
    L = dq.lib()
    assert L.snake_state_bytes(0) == dq.DQN_EINVAL
    assert L.snake_state_bytes(3) == 3 * dq.SNAKE_STATE_BYTES
    assert L.snake_reset(None, 4, FAKE, FAKE, None, None) == dq.DQN_EINVAL
    assert L.snake_reset(FAKE, 0, FAKE, FAKE, None, None) == dq.DQN_EINVAL
    assert L.snake_reset(FAKE + 8, 4, FAKE, FAKE, None, None) == dq.DQN_EINVAL      # misaligned games
    rp = native._CReplayOut()
    rp.frames, rp.action, rp.reward, rp.terminal = FAKE, FAKE, FAKE, FAKE
    rp.record_stride, rp.capacity = 28224, 1                                        # capacity < 2
    assert L.snake_reset(FAKE, 4, FAKE, FAKE, ctypes.byref(rp), None) == dq.DQN_EINVAL
    rp.capacity, rp.record_stride = 8, 28220                                        # stride not a multiple of 16
    assert L.snake_reset(FAKE, 4, FAKE, FAKE, ctypes.byref(rp), None) == dq.DQN_EINVAL
    rp.record_stride = 28224
    assert L.snake_step(FAKE, 4, FAKE, FAKE, FAKE, FAKE, FAKE, ctypes.byref(rp), -1, None) == dq.DQN_EINVAL
    assert L.snake_step(FAKE, 4, None, FAKE, FAKE, FAKE, FAKE, None, 0, None) == dq.DQN_EINVAL
    assert dq.dqn_anneal_epsilon(0, 100, 0.1, 1.0) == 1.0
    assert dq.dqn_anneal_epsilon(250, 100, 0.1, 1.0) == 0.1


@fake_ptr_test
def test_preprocess_argument_errors():
    L = dq.lib()
    OUT = FAKE + 2**32
    ok = dict(rgb=FAKE, n=4, h=176, w=176, top=4, left=4, f=2, out=OUT, stride=7056)

    def pre(**kw):
        a = {**ok, **kw}
        return L.dqn_preprocess(a["rgb"], a["n"], a["h"], a["w"], a["top"], a["left"], a["f"], a["out"],
                                a["stride"], None)
    assert pre(n=0) == dq.DQN_OK                                    # nothing to do
    assert pre(n=0, rgb=None, out=None) == dq.DQN_OK
    assert pre(rgb=None) == dq.DQN_EINVAL
    assert pre(out=None) == dq.DQN_EINVAL
    assert pre(n=-1) == dq.DQN_EINVAL
    for f in (0, 9):
        assert pre(f=f, h=2000, w=2000) == dq.DQN_EINVAL           # factor outside 1..8
    assert pre(top=9) == dq.DQN_EINVAL                              # window past the bottom edge
    assert pre(left=9) == dq.DQN_EINVAL                             # past the right edge
    assert pre(top=-1) == dq.DQN_EINVAL
    assert pre(rgb=FAKE + 4) == dq.DQN_EINVAL                      # rgb not 16-byte aligned
    assert pre(out=OUT + 4) == dq.DQN_EINVAL                       # out not 16-byte aligned
    assert pre(stride=7040) == dq.DQN_EINVAL                       # stride < 84*84
    assert pre(stride=7064) == dq.DQN_EINVAL                       # stride not a multiple of 16
    assert pre(out=FAKE + 4096) == dq.DQN_EINVAL                   # out overlaps rgb


@fake_ptr_test
def test_observe_argument_errors():
    L = dq.lib()
    ST = FAKE + 2**32
    rp = native._CReplayOut()
    rp.frames, rp.action, rp.reward, rp.terminal = FAKE + 2**33, FAKE + 2**34, FAKE + 2**34 + 4096, FAKE + 2**35
    rp.record_stride, rp.capacity = 28224, 16

    def obs(n=4, states=ST, actions=FAKE + 2**36, rewards=FAKE + 2**37, terminal=FAKE + 2**38, replay=rp, t=3,
            top=4, f=2, rgb=FAKE):
        return L.dqn_observe(rgb, n, 176, 176, top, 4, f, actions, rewards, terminal, states,
                             ctypes.byref(replay) if replay is not None else None, t, None)
    assert obs(n=0) == dq.DQN_EINVAL
    assert obs(t=-2) == dq.DQN_EINVAL
    assert obs(states=None) == dq.DQN_EINVAL
    assert obs(states=ST + 8) == dq.DQN_EINVAL                      # states not 16-byte aligned
    assert obs(terminal=None) == dq.DQN_EINVAL                      # t >= 0 needs the terminal flags
    assert obs(actions=None) == dq.DQN_EINVAL                       # ... and, with a replay, actions
    assert obs(rewards=None) == dq.DQN_EINVAL                       # ... and rewards
    assert obs(top=9) == dq.DQN_EINVAL
    assert obs(f=9) == dq.DQN_EINVAL
    assert obs(states=FAKE + 1024) == dq.DQN_EINVAL                 # states overlap the screens
    rp.capacity = 1
    assert obs() == dq.DQN_EINVAL                                   # replay capacity < 2
    rp.capacity, rp.record_stride = 16, 28200
    assert obs() == dq.DQN_EINVAL                                   # record stride too small


def test_status_strings():
    for s in (dq.DQN_OK, dq.DQN_EINVAL, dq.DQN_EWORKSPACE, dq.DQN_EHIP, dq.DQN_EUNSUPPORTED):
        assert dq.dqn_status_string(s) not in ("", "unknown status")


@fake_ptr_test
def test_td_gradient_replay_argument_errors():
    L = dq.lib()
    n = dq.NET_SMALL
    ws = dq.dqn_workspace_bytes(n, 8, dq.DQN_OP_TD_GRADIENT)
    rp = native._CReplay()
    rp.frames, rp.action, rp.reward, rp.terminal = FAKE, FAKE, FAKE, FAKE
    rp.record_stride, rp.size, rp.c, rp.h, rp.w = 28224, 100, 4, 84, 84

    def call(idx=FAKE, B=8, wsb=ws, **kw):
        for k, v in kw.items():
            setattr(rp, k, v)
        return L.dqn_td_gradient_replay(_cnet(n), FAKE, FAKE, ctypes.byref(rp), idx, B,
                                        ctypes.c_float(0.99), FAKE + 2**33, FAKE, None, None,
                                        FAKE + 2**34, wsb, None)
    assert call(idx=None) == dq.DQN_EINVAL
    assert call(B=0) == dq.DQN_EINVAL
    assert call(wsb=ws - 1) == dq.DQN_EWORKSPACE
    assert call(c=2) == dq.DQN_EINVAL                  # record shape differs from the input
    rp.c = 4
    assert call(size=1) == dq.DQN_EINVAL               # needs two records for s'
    rp.size = 100
    assert call(record_stride=28230) == dq.DQN_EINVAL
    rp.record_stride = 28224
    rp.action = None
    assert call() == dq.DQN_EINVAL                     # side arrays required


@fake_ptr_test
def test_forward_replay_argument_errors():
    L = dq.lib()
    n = dq.NET_LARGE
    ws = dq.dqn_workspace_bytes(n, 8, dq.DQN_OP_FORWARD)
    rp = native._CReplay()
    rp.frames, rp.action, rp.reward, rp.terminal = FAKE, None, None, None
    rp.record_stride, rp.size, rp.c, rp.h, rp.w = 28224, 100, 4, 84, 84

    def call(idx=FAKE, B=8, eps=0.0, draws=None, wsb=ws, **kw):
        for k, v in kw.items():
            setattr(rp, k, v)
        return L.dqn_forward_replay(_cnet(n), FAKE, ctypes.byref(rp), idx, B, ctypes.c_float(eps), draws,
                                    None, None, FAKE + 2**34, wsb, None)
    assert call(idx=None) == dq.DQN_EINVAL
    assert call(B=0) == dq.DQN_EINVAL
    assert call(wsb=ws - 1) == dq.DQN_EWORKSPACE
    assert call(eps=1.5) == dq.DQN_EINVAL
    assert call(eps=0.05) == dq.DQN_EINVAL             # exploring needs draws
    assert call(c=2) == dq.DQN_EINVAL                  # record shape differs from the input
    rp.c = 4
    assert call(size=0) == dq.DQN_EINVAL
    rp.size = 1                                        # one record is a valid state
    assert call(record_stride=28230) == dq.DQN_EINVAL
    rp.record_stride = 28224
    assert L.dqn_forward_replay(_cnet(n), FAKE, None, FAKE, 8, ctypes.c_float(0.0), None, None, None,
                                FAKE + 2**34, ws, None) == dq.DQN_EINVAL


@pytest.mark.parametrize("net,limit", [(dq.NET_SMALL, 289), (dq.NET_LARGE, 100), (dq.NET_LARGE_BF16, 93)])
def test_noalloc_batch_limits_match_the_header(net, limit):
    """dqn_td_gradient_noalloc runs in a 64 MiB static workspace: every batch
    up to the limit that include/dqn.h states fits it, the next does not."""
    cap = 64 * 2**20
    sizes = [dq.dqn_workspace_bytes(net, b, dq.DQN_OP_TD_GRADIENT) for b in range(1, limit + 2)]
    assert all(0 < s <= cap for s in sizes[:limit])
    assert sizes[limit] > cap
