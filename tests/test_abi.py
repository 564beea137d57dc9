"""Host-side checks of the C ABI (no GPU needed): the library loads, exports
every function include/specblock.h declares, and rejects invalid arguments
with the documented codes before enqueueing any device work."""
import ctypes as C
import os
import re

import pytest

from paper_2605_07243_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "specblock.h")


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(B.LIB_PATH):
        from paper_2605_07243_amd import build
        build.build()
    return B.load()


def header_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(sb_[a-z_]+)\s*\(", text)))


def test_exports_every_declared_function(lib):
    names = header_functions()
    assert "sb_draft_block_expand" in names and "sb_tree_verify" in names
    assert set(names) == set(B.EXPORTS)
    for n in names:
        assert hasattr(lib, n), n


def cfg(**kw):
    c = B.Config()
    c.target = B.ModelDims(2, 256, 4, 4, 64, 1024, 1024, 500000.0, 1e-5)
    c.drafter_layers = 1
    c.tap_layers[:] = [0, 1, 1]
    c.K, c.M, c.B_max, c.budget = 4, 3, 4, 32
    c.branch_map[:] = [2, 4, 6, 4]
    c.dtype = B.SB_F32
    c.max_seqs, c.page_size, c.max_pages, c.prefill_chunk = 1, 16, 16, 128
    for k, v in kw.items():
        if k.startswith("t_"):
            setattr(c.target, k[2:], v)
        else:
            setattr(c, k, v)
    return c


@pytest.mark.parametrize("kw,code", [
    (dict(dtype=7), B.SB_EDTYPE),
    (dict(t_head_dim=96), B.SB_ESHAPE),
    (dict(t_n_kv_heads=3), B.SB_ESHAPE),
    (dict(t_d_model=250), B.SB_ESHAPE),
    (dict(t_vocab=1000), B.SB_ESHAPE),
    (dict(K=0), B.SB_EINVAL),
    (dict(B_max=65), B.SB_EINVAL),
    (dict(budget=513), B.SB_EBUDGET),
    (dict(page_size=32), B.SB_ESHAPE),
    (dict(prefill_chunk=100), B.SB_EINVAL),
    (dict(max_seqs=0), B.SB_EINVAL),
    (dict(max_pages=0), B.SB_EINVAL),
    (dict(max_pages=16385), B.SB_EINVAL),
    (dict(tap_layers=(C.c_int32 * 3)(0, 1, 2)), B.SB_ESHAPE),
    (dict(t_rope_theta=0.0), B.SB_EINVAL),
    # bf16 projections: input widths % 128, output widths % 32
    (dict(dtype=B.SB_BF16, t_d_ff=1056), B.SB_ESHAPE),
    (dict(dtype=B.SB_BF16, t_d_model=288), B.SB_ESHAPE),
    (dict(dtype=B.SB_BF16, t_vocab=1040), B.SB_ESHAPE),
    # reduced drafter vocabulary: 10..vocab, multiple of 16 (bf16: of 32)
    (dict(draft_vocab=8), B.SB_ESHAPE),
    (dict(draft_vocab=1040), B.SB_ESHAPE),
    (dict(draft_vocab=1000), B.SB_ESHAPE),
    (dict(dtype=B.SB_BF16, draft_vocab=528), B.SB_ESHAPE),
    # head updates: at most 64 positions; drafter vocabulary % 64, d % CW
    (dict(adapt_cap=65), B.SB_EINVAL),
    (dict(adapt_cap=-1), B.SB_EINVAL),
    (dict(adapt_cap=8, draft_vocab=528), B.SB_ESHAPE),
])
def test_create_rejects_bad_configs(lib, kw, code):
    c = cfg(**kw)
    ctx = C.c_void_p()
    assert lib.sb_create(C.byref(c), C.byref(ctx)) == code
    assert not ctx.value
    assert lib.sb_last_error(None)
    assert lib.sb_workspace_bytes(C.byref(c)) == 0


def test_capacities(lib):
    c = cfg()
    assert lib.sb_row_capacity(C.byref(c)) == 4 + 2 * 4 * 4
    assert lib.sb_workspace_bytes(C.byref(c)) > 0


class Fake:
    """Aligned, never-dereferenced addresses (host tests enqueue nothing)."""

    def __init__(self):
        self.buf = (C.c_char * (1 << 16))()
        base = C.addressof(self.buf)
        self.p = C.c_void_p((base + 255) & ~255)

    def at(self, off=0):
        return C.c_void_p(self.p.value + off)


@pytest.fixture
def bound(lib):
    c = cfg()
    ctx = C.c_void_p()
    assert lib.sb_create(C.byref(c), C.byref(ctx)) == B.SB_OK
    f = Fake()
    layers = (B.LayerWeights * 2)(*[B.LayerWeights(*[f.at()] * 6, None)
                                    for _ in range(2)])
    dl = (B.LayerWeights * 1)(B.LayerWeights(*[f.at()] * 7))
    tw = B.TargetWeights(f.at(), layers, f.at(), f.at())
    dw = B.DrafterWeights(f.at(), f.at(), f.at(), f.at(), f.at(), f.at(), dl,
                          f.at(), f.at(), f.at(), f.at(), None)
    need = lib.sb_workspace_bytes(C.byref(c))
    # too small, misaligned, then right: none of these touches the device
    assert lib.sb_bind(ctx, C.byref(tw), C.byref(dw), f.at(), need - 1) == \
        B.SB_EBUDGET
    assert lib.sb_bind(ctx, C.byref(tw), C.byref(dw), f.at(8), need) == \
        B.SB_EINVAL
    bad = B.DrafterWeights(f.at(8), *([f.at()] * 5), dl, *([f.at()] * 4))
    assert lib.sb_bind(ctx, C.byref(tw), C.byref(bad), f.at(), need) == \
        B.SB_EINVAL     # bf16/fp32 matrices need 16-byte alignment
    nos = (B.LayerWeights * 1)(B.LayerWeights(*[f.at()] * 6, None))
    dw2 = B.DrafterWeights(*([f.at()] * 6), nos, *([f.at()] * 4))
    assert lib.sb_bind(ctx, C.byref(tw), C.byref(dw2), f.at(), need) == \
        B.SB_EINVAL     # drafter layers need W_shift
    assert lib.sb_bind(ctx, C.byref(tw), C.byref(dw), f.at(), need) == B.SB_OK
    yield lib, ctx, f
    lib.sb_destroy(ctx)


def test_calls_before_bind_are_refused(lib):
    c = cfg()
    ctx = C.c_void_p()
    assert lib.sb_create(C.byref(c), C.byref(ctx)) == B.SB_OK
    t = B.Tree()
    assert lib.sb_accept(ctx, 1, C.byref(t), None, None, None) == B.SB_ESTATE
    # the debug status word lives in the workspace
    assert lib.sb_set_debug(ctx, 1) == B.SB_ESTATE
    assert lib.sb_device_check(ctx, None) == B.SB_ESTATE
    assert lib.sb_set_debug(None, 1) == B.SB_EINVAL
    assert lib.sb_device_check(None, None) == B.SB_EINVAL
    lib.sb_destroy(ctx)


def _tree(f):
    return B.Tree(*[f.at() for _ in B.TREE_FIELDS])


def test_draft_call_validation(bound):
    lib, ctx, f = bound
    seqs = B.Seqs(1, f.at(), f.at(), f.at())
    kv = B.KV(f.at(), f.at(), f.at(), 1, 4)
    tree = _tree(f)
    out = B.DraftOut(*[f.at() for _ in B.DRAFT_OUT_FIELDS])
    call = lambda m, K, s=seqs, k=kv, t=tree, o=out: lib.sb_draft_block_expand(  # noqa
        ctx, m, K, C.byref(s), C.byref(k), C.byref(t), C.byref(o), None)
    assert call(1, 3) == B.SB_ESHAPE                   # K != cfg.K
    assert call(0, 4) == B.SB_EINVAL                   # block index
    assert call(4, 4) == B.SB_EINVAL                   # > M
    assert call(1, 4, s=B.Seqs(2, f.at(), f.at(), f.at())) == B.SB_ESHAPE
    assert call(1, 4, k=B.KV(f.at(), f.at(), f.at(), 2, 4)) == B.SB_ESHAPE
    t2 = _tree(f)
    t2.anc = None
    assert call(1, 4, t=t2) == B.SB_EINVAL
    o2 = B.DraftOut(*[f.at() for _ in B.DRAFT_OUT_FIELDS])
    o2.logits = f.at(4)
    assert call(1, 4, o=o2) == B.SB_EINVAL
    assert b"logits" in lib.sb_last_error(ctx)


def test_verify_accept_commit_validation(bound):
    lib, ctx, f = bound
    seqs = B.Seqs(1, f.at(), f.at(), f.at())
    tkv = B.KV(f.at(), f.at(), f.at(), 2, 4)
    dkv = B.KV(f.at(), f.at(), f.at(), 1, 4)
    tree = _tree(f)
    v = B.VerifyOut(None, f.at(), None)
    assert lib.sb_tree_verify(ctx, C.byref(seqs), C.byref(tree),
                              C.byref(tkv), C.byref(v), None) == B.SB_EINVAL
    v = B.VerifyOut(f.at(), f.at(), None)
    assert lib.sb_tree_verify(ctx, C.byref(seqs), C.byref(tree),
                              C.byref(dkv), C.byref(v), None) == B.SB_ESHAPE
    a = B.AcceptOut(f.at(), f.at(), None)
    assert lib.sb_accept(ctx, 1, C.byref(tree), f.at(), C.byref(a),
                         None) == B.SB_EINVAL
    assert lib.sb_accept(ctx, 2, C.byref(tree), f.at(), C.byref(a),
                         None) == B.SB_ESHAPE
    a = B.AcceptOut(f.at(), f.at(), f.at())
    assert lib.sb_commit(ctx, C.byref(seqs), C.byref(tree), C.byref(v),
                         C.byref(a), C.byref(dkv), C.byref(dkv),
                         None) == B.SB_ESHAPE
    lens = (C.c_int32 * 1)(0)
    assert lib.sb_prefill(ctx, C.byref(seqs), f.at(), 8, lens, C.byref(tkv),
                          C.byref(dkv), None) == B.SB_ESHAPE
    lens = (C.c_int32 * 1)(300)
    assert lib.sb_prefill(ctx, C.byref(seqs), f.at(), 400, lens, C.byref(tkv),
                          C.byref(dkv), None) == B.SB_EBUDGET
    assert lib.sb_set_length_bound(ctx, -1) == B.SB_EINVAL


def test_create_accepts_bf16_shapes(lib):
    c = cfg(dtype=B.SB_BF16)
    ctx = C.c_void_p()
    assert lib.sb_create(C.byref(c), C.byref(ctx)) == B.SB_OK
    lib.sb_destroy(ctx)


@pytest.mark.parametrize("args,code", [
    # src, dst, rows, cols, dtype, gate_up (fake, never dereferenced: every
    # case fails validation before anything is enqueued)
    ((0x10000, 0x90000, 64, 128, 7, 0), B.SB_EDTYPE),
    ((0x10000, 0x90000, 0, 128, B.SB_BF16, 0), B.SB_EINVAL),
    ((0x10000, 0x90000, 64, -1, B.SB_BF16, 0), B.SB_EINVAL),
    ((0, 0x90000, 64, 128, B.SB_BF16, 0), B.SB_EINVAL),
    ((0x10008, 0x90000, 64, 128, B.SB_BF16, 0), B.SB_EINVAL),
    ((0x10000, 0x12000, 64, 128, B.SB_BF16, 0), B.SB_EINVAL),   # overlap
    ((0x10000, 0x90000, 48, 128, B.SB_BF16, 0), B.SB_ESHAPE),
    ((0x10000, 0x90000, 64, 96, B.SB_BF16, 1), B.SB_ESHAPE),
])
def test_pack_weight_validation(lib, args, code):
    src, dst, rows, cols, dtype, gate_up = args
    assert lib.sb_pack_weight(C.c_void_p(src), C.c_void_p(dst), rows, cols,
                              dtype, gate_up, None) == code
    assert lib.sb_last_error(None)


def test_reduced_vocab_needs_map(lib):
    c = cfg(draft_vocab=512)
    ctx = C.c_void_p()
    assert lib.sb_create(C.byref(c), C.byref(ctx)) == B.SB_OK
    f = Fake()
    layers = (B.LayerWeights * 2)(*[B.LayerWeights(*[f.at()] * 6, None)
                                    for _ in range(2)])
    dl = (B.LayerWeights * 1)(B.LayerWeights(*[f.at()] * 7))
    tw = B.TargetWeights(f.at(), layers, f.at(), f.at())
    dw = B.DrafterWeights(*([f.at()] * 6), dl, *([f.at()] * 4), None)
    need = lib.sb_workspace_bytes(C.byref(c))
    assert lib.sb_bind(ctx, C.byref(tw), C.byref(dw), f.at(), need) == \
        B.SB_EINVAL
    assert b"d2t" in lib.sb_last_error(ctx)
    lib.sb_destroy(ctx)


def test_struct_layouts_match_header(tmp_path):
    """Every ctypes structure has the size and field offsets that a C
    compiler gives the header's struct."""
    import shutil
    import subprocess
    cc = shutil.which("gcc") or shutil.which("cc")
    if cc is None:
        pytest.skip("no C compiler")
    structs = {"sb_model_dims": B.ModelDims, "sb_config": B.Config,
               "sb_layer_weights": B.LayerWeights,
               "sb_target_weights": B.TargetWeights,
               "sb_drafter_weights": B.DrafterWeights, "sb_kv": B.KV,
               "sb_seqs": B.Seqs, "sb_tree": B.Tree, "sb_draft_out": B.DraftOut,
               "sb_verify_out": B.VerifyOut, "sb_accept_out": B.AcceptOut,
               "sb_kernel_stat": B.KernelStat, "sb_gemm_stat": B.GemmStat,
               "sb_adapt_buffer": B.AdaptBuffer,
               "sb_head_weights": B.HeadWeights}
    lines = ['#include <stdio.h>', '#include <stddef.h>',
             f'#include "{HEADER}"', 'int main(void) {']
    for cname, py in structs.items():
        lines.append(f'printf("{cname} %zu\\n", sizeof({cname}));')
        for fname, _ in py._fields_:
            lines.append(f'printf("{cname}.{fname} %zu\\n", '
                         f'offsetof({cname}, {fname}));')
    lines.append("return 0; }")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run([cc, str(src), "-o", str(exe)], check=True)
    got = dict(l.split() for l in
               subprocess.run([str(exe)], check=True, capture_output=True,
                              text=True).stdout.splitlines())
    for cname, py in structs.items():
        assert int(got[cname]) == C.sizeof(py), cname
        for fname, _ in py._fields_:
            assert int(got[f"{cname}.{fname}"]) == getattr(py, fname).offset, \
                (cname, fname)


def test_accept_sample_validation(bound):
    lib, ctx, f = bound
    tree = _tree(f)
    out = B.AcceptOut(f.at(), f.at(), f.at())
    call = lambda n=1, z=f.at(), T=1.0, ua=f.at(), ub=f.at(), o=out: \
        lib.sb_accept_sample(ctx, n, C.byref(tree), z, T, ua, ub,  # noqa
                             C.byref(o), None)
    assert call(T=0.0) == B.SB_EINVAL
    assert call(T=-1.0) == B.SB_EINVAL
    assert call(T=float("inf")) == B.SB_EINVAL
    assert call(T=float("nan")) == B.SB_EINVAL
    assert b"temperature" in lib.sb_last_error(ctx)
    assert call(z=None) == B.SB_EINVAL
    assert call(ua=f.at(2)) == B.SB_EINVAL
    assert call(o=B.AcceptOut(f.at(), None, f.at())) == B.SB_EINVAL
    assert call(o=B.AcceptOut(f.at(), f.at(), f.at(), f.at(2))) == B.SB_EINVAL
    assert call(n=0) == B.SB_ESHAPE
    assert call(n=2) == B.SB_ESHAPE


def test_adaptation_validation(bound):
    lib, ctx, f = bound
    tree = _tree(f)
    acc = B.AcceptOut(f.at(), f.at(), f.at())
    buf = B.AdaptBuffer(f.at(), f.at(), f.at(), 8)
    hw = B.HeadWeights(f.at(256), f.at(), f.at())
    # the bound context has adapt_cap 0
    assert lib.sb_adapt_push(ctx, 1, C.byref(tree), C.byref(acc),
                             C.byref(buf), None) == B.SB_ESTATE
    assert lib.sb_head_update(ctx, C.byref(buf), f.at(512), C.byref(hw), 0.1,
                              0.01, None, None) == B.SB_ESTATE
    assert b"adapt_cap" in lib.sb_last_error(ctx)


def test_adaptation_argument_checks(lib):
    c = cfg(adapt_cap=8)
    ctx = C.c_void_p()
    assert lib.sb_create(C.byref(c), C.byref(ctx)) == B.SB_OK
    f = Fake()
    layers = (B.LayerWeights * 2)(*[B.LayerWeights(*[f.at()] * 6, None)
                                    for _ in range(2)])
    dl = (B.LayerWeights * 1)(B.LayerWeights(*[f.at()] * 7))
    tw = B.TargetWeights(f.at(), layers, f.at(), f.at())
    dw = B.DrafterWeights(*([f.at()] * 6), dl, *([f.at()] * 4), None)
    need = lib.sb_workspace_bytes(C.byref(c))
    ws = (C.c_char * (need + 512))()
    wp = C.c_void_p((C.addressof(ws) + 255) & ~255)
    assert lib.sb_bind(ctx, C.byref(tw), C.byref(dw), wp, need) == B.SB_OK
    tree = _tree(f)
    acc = B.AcceptOut(f.at(), f.at(), f.at())
    ok_buf = B.AdaptBuffer(f.at(), f.at(), f.at(), 8)
    push = lambda n=1, b=ok_buf: lib.sb_adapt_push(  # noqa: E731
        ctx, n, C.byref(tree), C.byref(acc), C.byref(b), None)
    assert push(b=B.AdaptBuffer(f.at(), f.at(), f.at(), 4)) == B.SB_ESHAPE
    assert push(b=B.AdaptBuffer(f.at(), None, f.at(), 8)) == B.SB_EINVAL
    assert push(n=0) == B.SB_ESHAPE
    upd = lambda hw, lr=0.1, kl=0.01, w0=f.at(512): lib.sb_head_update(  # noqa
        ctx, C.byref(ok_buf), w0, C.byref(hw), lr, kl, None, None)
    good = B.HeadWeights(f.at(256), f.at(), f.at())
    assert upd(good, lr=-1.0) == B.SB_EINVAL
    assert upd(good, kl=float("nan")) == B.SB_EINVAL
    assert upd(good, w0=f.at(256)) == B.SB_EINVAL       # same as train
    assert upd(B.HeadWeights(f.at(), f.at(), f.at())) == B.SB_EINVAL  # bound
    assert upd(B.HeadWeights(f.at(8), f.at(), f.at())) == B.SB_EINVAL
    lib.sb_destroy(ctx)


def _fake_tree():
    """A tree whose every pointer is non-NULL and aligned host memory: the
    calls below must fail their host-side checks before touching it."""
    buf = (C.c_int32 * 64)()
    p = C.cast(buf, C.c_void_p)
    t = B.Tree(*([p] * len(B.Tree._fields_)))
    return t, buf


def test_noalloc_accept_rejects_sizes_past_its_static_scratch(lib):
    """sb_accept_sample_noalloc keeps n_seqs * budget * ceil(vocab / 16384)
    tile statistics in a static array of 65536 entries: 8 x 512 x 16 fits
    exactly, 9 sequences do not (SB_EBUDGET, before any device work); the
    signal r needs a bound context (SB_ESTATE)."""
    c = cfg(t_vocab=262144, budget=512, max_seqs=16)
    ctx = C.c_void_p()
    assert lib.sb_create(C.byref(c), C.byref(ctx)) == B.SB_OK
    try:
        t, keep = _fake_tree()
        buf = (C.c_float * 64)()
        fp = C.cast(buf, C.c_void_p)
        out = B.AcceptOut(fp, fp, fp, None)
        rc = lib.sb_accept_sample_noalloc(ctx, 9, C.byref(t), fp, 1.0, fp, fp,
                                          C.byref(out), None)
        assert rc == B.SB_EBUDGET
        assert b"65536" in lib.sb_last_error(ctx)
        out_r = B.AcceptOut(fp, fp, fp, fp)
        rc = lib.sb_accept_sample_noalloc(ctx, 1, C.byref(t), fp, 1.0, fp, fp,
                                          C.byref(out_r), None)
        assert rc == B.SB_ESTATE
        rc = lib.sb_accept_sample_noalloc(ctx, 1, C.byref(t), fp, 0.0, fp, fp,
                                          C.byref(out), None)
        assert rc == B.SB_EINVAL
        rc = lib.sb_accept_sample_noalloc(ctx, 17, C.byref(t), fp, 1.0, fp,
                                          fp, C.byref(out), None)
        assert rc == B.SB_ESHAPE
    finally:
        lib.sb_destroy(ctx)
