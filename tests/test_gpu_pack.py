"""sb_pack_weight on the GPU: the packed bf16 layout is exactly the
permutation the header defines (checked against an index formula written
here from that definition), with and without the gate/up interleave, and
f32 weights are copied unchanged."""
import ctypes as C

import numpy as np
import pytest
import torch

from paper_2605_07243_amd import binding as B

pytestmark = pytest.mark.gpu


def expected_packed(src: np.ndarray, gate_up: bool) -> np.ndarray:
    rows, cols = src.shape
    idx = np.arange(rows * cols)
    e = idx % 8
    lane = (idx // 8) % 64
    i = (idx // 512) % 4
    blk = idx // 2048
    kb, rb = blk // (rows // 32), blk % (rows // 32)
    j = lane % 32
    if gate_up:
        row = np.where(j < 16, 16 * rb + j, rows // 2 + 16 * rb + j - 16)
    else:
        row = 32 * rb + j
    col = 64 * kb + 32 * (lane // 32) + 8 * i + e
    return src[row, col]


def pack(lib, t, dtype, gate_up):
    out = torch.empty_like(t)
    rc = lib.sb_pack_weight(C.c_void_p(t.data_ptr()), C.c_void_p(out.data_ptr()),
                            t.shape[0], t.shape[1], dtype, int(gate_up), None)
    assert rc == B.SB_OK, lib.sb_last_error(None)
    torch.cuda.synchronize()
    return out


@pytest.mark.parametrize("rows,cols,gate_up", [
    (32, 64, False), (96, 192, False), (4096 + 32, 384, False),
    (64, 128, True), (3072, 512, True)])
def test_pack_bf16_layout(rows, cols, gate_up):
    lib = B.load()
    g = torch.Generator(device="cuda").manual_seed(rows * 7 + cols)
    t = torch.randn(rows, cols, generator=g, device="cuda").to(torch.bfloat16)
    got = pack(lib, t, B.SB_BF16, gate_up).view(torch.int16).cpu().numpy()
    src = t.view(torch.int16).cpu().numpy()
    want = expected_packed(src, gate_up)
    assert np.array_equal(got.reshape(-1), want)


def test_pack_f32_is_a_copy():
    lib = B.load()
    t = torch.randn(40, 24, device="cuda")
    got = pack(lib, t, B.SB_F32, False)
    assert torch.equal(got, t)
