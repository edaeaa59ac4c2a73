"""C-ABI checks that need no GPU: the library loads, exports every declared
symbol, and rejects bad arguments before touching HIP."""
import ctypes as C
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "tandem.h")

L = pytest.importorskip("paper_2606_28166_amd._lib", reason="libtandem.so not built")

import workloads as W  # noqa: E402
from paper_2606_28166_amd.engine import model_cfg  # noqa: E402


def _declared():
    txt = open(HEADER).read()
    return sorted(set(re.findall(r"\b(tandem_[a-z_]+)\s*\(", txt)))


def test_header_symbols_are_exported():
    names = _declared()
    assert "tandem_init" in names and "tandem_step" in names
    for n in names:
        assert hasattr(L.lib, n), n
    assert set(L.EXPORTS) == set(names)


def _cfgs(name="small"):
    wl = W.workload(name)
    return model_cfg(wl.senior), model_cfg(wl.junior)


def test_workspace_size_matches_layout():
    s, j = _cfgs("qwen")
    cap = L.Capacity(128, 256 - 1 + 2048, 4096)
    kv, sc = L.tandem_workspace_size(s, j, cap)
    ctx = ((2303 + 63) // 64) * 64
    want_kv = 2 * 2 * 128 * ctx * 128 * 8 * (36 + 28)
    assert kv == want_kv
    assert sc > 128 * 151936 * 4 * 2


@pytest.mark.parametrize("mut,code", [
    (lambda s, j: setattr(j, "vocab", s.vocab + 1), L.E_SHAPE),
    (lambda s, j: setattr(s, "head_dim", 96), L.E_UNSUPPORTED),
    (lambda s, j: setattr(s, "n_kv_heads", 3), L.E_SHAPE),
    (lambda s, j: setattr(j, "weight_dtype", 7), L.E_ARG),
    (lambda s, j: setattr(s, "d_model", 0), L.E_SHAPE),
])
def test_workspace_size_rejects_bad_shapes(mut, code):
    s, j = _cfgs()
    mut(s, j)
    kv, sc = C.c_size_t(), C.c_size_t()
    cap = L.Capacity(8, 64, 64)
    st = L.lib.tandem_workspace_size(C.byref(s), C.byref(j), C.byref(cap), C.byref(kv), C.byref(sc))
    assert st == code
    assert L.lib.tandem_last_error(None)


def test_capacity_and_null_checks():
    s, j = _cfgs()
    kv, sc = C.c_size_t(), C.c_size_t()
    cap = L.Capacity(0, 64, 64)
    assert L.lib.tandem_workspace_size(C.byref(s), C.byref(j), C.byref(cap), C.byref(kv), C.byref(sc)) == L.E_CAPACITY
    assert L.lib.tandem_workspace_size(None, C.byref(j), C.byref(cap), C.byref(kv), C.byref(sc)) == L.E_ARG


def _fake_model(cfg, fill=0x1000):
    n = cfg.n_layers * 8
    ptrs = (C.c_void_p * n)(*([fill] * n))
    m = L.Model(cfg, fill, C.cast(ptrs, C.POINTER(C.c_void_p)), fill, fill)
    return m, ptrs


def _init(sen_cfg, jun_cfg, sw=None, smp=None, cap=None, kv_bytes=None, sc_bytes=None, kv_ptr=0x10000,
          sc_ptr=0x20000):
    cap = cap or L.Capacity(8, 64, 64)
    ms, ps = _fake_model(sen_cfg)
    mj, pj = _fake_model(jun_cfg)
    sw = sw or L.SwitchCfg(L.SWITCH, 0.1, -1, None, L.SENIOR)
    smp = smp or L.SampleCfg(1.0, -1, 0.0, 0.0, 16, 7)
    out = L.Outputs(0x3000, 0x3000, 0x3000, 0x3000)
    need_kv, need_sc = C.c_size_t(), C.c_size_t()
    L.lib.tandem_workspace_size(C.byref(sen_cfg), C.byref(jun_cfg), C.byref(cap), C.byref(need_kv), C.byref(need_sc))
    h = C.c_void_p()
    st = L.lib.tandem_init(C.byref(ms), C.byref(mj), C.byref(sw), C.byref(smp), C.byref(cap), kv_ptr,
                           kv_bytes if kv_bytes is not None else need_kv.value, sc_ptr,
                           sc_bytes if sc_bytes is not None else need_sc.value, C.byref(out), None, C.byref(h))
    return st, h


def test_init_rejects_bad_arguments_before_hip():
    s, j = _cfgs()
    j2 = L.ModelCfg.from_buffer_copy(j)
    j2.vocab = s.vocab - 1
    assert _init(s, j2)[0] == L.E_SHAPE
    assert _init(s, j, sw=L.SwitchCfg(L.SWITCH, 1.5, -1, None, L.SENIOR))[0] == L.E_ARG
    assert _init(s, j, sw=L.SwitchCfg(5, 0.5, -1, None, L.SENIOR))[0] == L.E_ARG
    assert _init(s, j, sw=L.SwitchCfg(L.SWITCH, 0.5, -1, None, 9))[0] == L.E_ARG
    assert _init(s, j, smp=L.SampleCfg(0.0, -1, 0, 0, 16, 1))[0] == L.E_ARG
    assert _init(s, j, smp=L.SampleCfg(1.0, s.vocab, 0, 0, 16, 1))[0] == L.E_ARG
    assert _init(s, j, smp=L.SampleCfg(1.0, -1, 0, 0, 100, 1))[0] == L.E_CAPACITY     # max_new > max_ctx
    assert _init(s, j, kv_bytes=16)[0] == L.E_CAPACITY
    assert _init(s, j, sc_bytes=16)[0] == L.E_CAPACITY
    assert _init(s, j, kv_ptr=0x10010)[0] == L.E_ARG                                  # misaligned
    # (never call init with valid arguments on fake pointers: it would launch kernels on them)


def test_null_handle_calls():
    assert L.lib.tandem_step(None, None) == L.E_ARG
    assert L.lib.tandem_prefill(None, None, None, 1, 1) == L.E_ARG
    assert L.lib.tandem_get_state(None, None, None, None, None, None) == L.E_ARG
    L.lib.tandem_destroy(None)
    assert L.lib.tandem_status_string(L.E_CAPACITY) == b"TANDEM_E_CAPACITY"


def test_grpo_workspace_size_and_argument_checks():
    cfg = L.GrpoCfg(16, 8, 3000, 0.2)
    # counts [128] int32, partials [128][ceil(3000 / 1024)] float and a ticket, each 256-aligned
    assert L.tandem_grpo_workspace_size(cfg) == 512 + 1536 + 256
    for bad, code in ((L.GrpoCfg(0, 8, 3000, 0.2), L.E_SHAPE), (L.GrpoCfg(16, 0, 3000, 0.2), L.E_SHAPE),
                      (L.GrpoCfg(16, 8, 0, 0.2), L.E_SHAPE), (L.GrpoCfg(1024, 8, 3000, 0.2), L.E_SHAPE),
                      (L.GrpoCfg(16, 8, 3000, 1.0), L.E_ARG), (L.GrpoCfg(16, 8, 3000, -0.1), L.E_ARG)):
        n = C.c_size_t()
        assert L.lib.tandem_grpo_workspace_size(C.byref(bad), C.byref(n)) == code
        assert L.lib.tandem_last_error(None)
    assert L.lib.tandem_grpo_workspace_size(C.byref(cfg), None) == L.E_ARG
    # every check fires before any HIP call: fake, never dereferenced addresses
    fake = 1 << 20
    ws = L.tandem_grpo_workspace_size(cfg)
    call = L.lib.tandem_grpo_loss
    assert call(None, fake, fake, fake, fake, None, fake, None, fake, fake, fake, ws, None) == L.E_ARG
    assert call(C.byref(cfg), None, fake, fake, fake, None, fake, None, fake, fake, fake, ws, None) == L.E_ARG
    assert call(C.byref(cfg), fake, fake, fake, fake, None, fake, None, None, fake, fake, ws, None) == L.E_ARG
    assert call(C.byref(cfg), fake, fake, fake, fake, None, fake, None, fake, fake, fake, ws - 1, None) == L.E_ARG
    assert call(C.byref(cfg), fake, fake, fake, fake, None, fake, None, fake, fake, fake + 16, ws, None) == L.E_ARG
    assert b"aligned" in L.lib.tandem_last_error(None)


def test_grpo_noalloc_argument_and_capacity_checks():
    # every check fires before any HIP call: fake, never dereferenced addresses
    fake = 1 << 20
    call = L.lib.tandem_grpo_loss_noalloc
    cfg = L.GrpoCfg(16, 8, 3000, 0.2)
    assert call(None, fake, fake, fake, fake, None, fake, None, fake, fake, None) == L.E_ARG
    assert call(C.byref(cfg), None, fake, fake, fake, None, fake, None, fake, fake, None) == L.E_ARG
    assert call(C.byref(cfg), fake, fake, fake, fake, None, fake, None, None, fake, None) == L.E_ARG
    assert call(C.byref(L.GrpoCfg(16, 8, 3000, 1.5)), fake, fake, fake, fake, None, fake, None, fake, fake,
                None) == L.E_ARG
    # the device array holds 1 MiB: 2^17 rollouts of 100 positions need
    # 512 KiB of counts + 512 KiB of partial sums + 256 bytes
    big = L.GrpoCfg(1 << 17, 1, 100, 0.2)
    assert L.tandem_grpo_workspace_size(big) == (1 << 20) + 256
    assert call(C.byref(big), fake, fake, fake, fake, None, fake, None, fake, fake, None) == L.E_CAPACITY
    assert b"holds 1048576" in L.lib.tandem_last_error(None)


def test_workspace_size_of_the_senior_alone():
    s, j = _cfgs("qwen")
    cap = L.Capacity(128, 256 - 1 + 2048, 4096)
    kv2, sc2 = L.tandem_workspace_size(s, j, cap)
    kv1, sc1 = L.tandem_workspace_size(s, None, cap)
    ctx = ((2303 + 63) // 64) * 64
    assert kv1 == 2 * 2 * 128 * ctx * 128 * 8 * 36          # the senior's K and V only
    assert kv1 < kv2 and sc1 < sc2


def _header_constants():
    """Integer constants the header defines in its enums: NAME = value, with
    values written as integers or as 1 << n."""
    txt = re.sub(r"/\*.*?\*/", "", open(HEADER).read(), flags=re.S)
    out = {}
    for name, val in re.findall(r"\b(TANDEM_[A-Z_0-9]+)\s*=\s*(-?\d+(?:\s*<<\s*\d+)?)", txt):
        a, _, b = val.partition("<<")
        out[name] = int(a) << int(b) if b else int(a)
    return out


def test_binding_constants_match_the_header():
    c = _header_constants()
    pairs = {"TANDEM_K_ATTENTION": L.K_ATTENTION, "TANDEM_K_GEMM": L.K_GEMM, "TANDEM_K_SAMPLE": L.K_SAMPLE,
             "TANDEM_K_OTHER": L.K_OTHER, "TANDEM_TIMING_SERIAL": L.TIMING_SERIAL,
             "TANDEM_TIMING_EAGER": L.TIMING_EAGER, "TANDEM_TIMING_SEPARATE_SAMPLE": L.TIMING_SEPARATE_SAMPLE,
             "TANDEM_E_ARG": L.E_ARG, "TANDEM_E_SHAPE": L.E_SHAPE, "TANDEM_E_CAPACITY": L.E_CAPACITY,
             "TANDEM_E_STATE": L.E_STATE, "TANDEM_E_HIP": L.E_HIP, "TANDEM_E_UNSUPPORTED": L.E_UNSUPPORTED}
    for name, val in pairs.items():
        assert c[name] == val, name
    # the mode flags sit above the class bits
    assert min(c["TANDEM_TIMING_SERIAL"], c["TANDEM_TIMING_EAGER"], c["TANDEM_TIMING_SEPARATE_SAMPLE"]) \
        >= 1 << c["TANDEM_K_CLASSES"]


def test_workspace_holds_the_lm_head_sampling_buffers_only_where_they_are_used():
    """Where both LM heads can sample in their GEMM epilogue (bf16, vocab a
    multiple of 4) the scratch holds the step's Gumbel noise for up to 128
    rows and the heads' per-workgroup partials; with a vocabulary that is not
    a multiple of 4 it holds neither."""
    s, j = _cfgs("small")
    cap = L.Capacity(64, 640, 256)
    _, sc = L.tandem_workspace_size(s, j, cap)
    s.vocab = j.vocab = 32001
    _, sc_odd = L.tandem_workspace_size(s, j, cap)
    noise = 64 * 32000 * 4
    parts = 2 * 64 * 1024 * 5 * 4
    # the odd vocabulary adds a logit per sequence per model and a 32-row block to each packed
    # LM head (d 1024 and 512), and loses the noise and the partials
    extra = 2 * 64 * 1 * 4 + 32 * (1024 + 512) * 2
    assert sc - sc_odd == pytest.approx(noise + parts - extra, abs=8 * 256)
    # the noise and partial rows stop at 128 sequences: 64 more sequences below
    # 128 add them, 64 more above 128 do not
    s, j = _cfgs("small")
    sc64, sc128, sc192 = (L.tandem_workspace_size(s, j, L.Capacity(n, 640, 64))[1] for n in (64, 128, 192))
    assert (sc128 - sc64) - (sc192 - sc128) == pytest.approx(64 * 32000 * 4 + 2 * 64 * 1024 * 5 * 4, abs=64 * 256)
