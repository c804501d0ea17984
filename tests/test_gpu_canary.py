"""Out-of-bounds writes: every output buffer of every entry point sits between guard
regions filled with a sentinel bit pattern, which must survive the call (ragged sizes,
aligned and misaligned starts). Values are checked by the parity tests; this checks
only that nothing is written outside the outputs, and that unused code bits are zero."""

import numpy as np
import pytest
import torch

import paper_2406_16282_amd as lmbp
from paper_2406_16282_amd import binding

pytestmark = pytest.mark.gpu
DEV = "cuda:0"
G = 256                      # guard elements on each side
SENT16, SENT32 = 0x5A5A, 0x5A5A5A5A


def guarded(n, dtype, off=0):
    """(buffer, view of n elements starting G + off elements in) with sentinel guards."""
    if dtype == torch.int32:
        buf = torch.full((n + 2 * G + off,), SENT32, dtype=torch.int32, device=DEV)
        return buf, buf[G + off:G + off + n]
    if dtype == torch.bfloat16:
        raw = torch.full((n + 2 * G + off,), SENT16, dtype=torch.int16, device=DEV)
    else:
        raw = torch.full((n + 2 * G + off,), SENT32, dtype=torch.int32, device=DEV)
    buf = raw.view(dtype)
    return buf, buf[G + off:G + off + n]


def check_guards(buf, n, off, what):
    torch.cuda.synchronize()
    raw = buf.view(torch.int16 if buf.element_size() == 2 else torch.int32).cpu().numpy()
    sent = SENT16 if buf.element_size() == 2 else SENT32
    sent = np.array(sent, dtype=raw.dtype)
    assert np.all(raw[:G + off] == sent), f"{what}: write before the buffer"
    assert np.all(raw[G + off + n:] == sent), f"{what}: write past the buffer"


def rnd(n, dtype, scale=2.0):
    return (torch.randn(n, device=DEV) * scale).to(dtype)


ACT_SIZES = [1, 15, 17, 1000, 5 * 4096 + 3, 65536 + 7]


@pytest.mark.parametrize("off", [0, 1])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("op", ["regelu2", "resilu2"])
def test_activation_guards(op, dtype, off):
    fwd, bwd = getattr(lmbp, op + "_fwd"), getattr(lmbp, op + "_bwd")
    for n in ACT_SIZES:
        words = binding.codes_words(n)
        x = rnd(n, dtype)
        yb, y = guarded(n, dtype, off)
        cb, c = guarded(words, torch.int32)
        fwd(x, y=y, codes=c)
        check_guards(yb, n, off, f"{op} y n={n}")
        check_guards(cb, words, 0, f"{op} codes n={n}")
        if n % 16:
            last = int(c[-1].item()) & 0xFFFFFFFF
            assert last >> (2 * (n % 16)) == 0, "unused code bits are not zero"
        db, dx = guarded(n, dtype, off)
        bwd(rnd(n, dtype), c, dx=dx)
        check_guards(db, n, off, f"{op} dx n={n}")


@pytest.mark.parametrize("off", [0, 1])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_swiglu_guards(dtype, off):
    for n in ACT_SIZES:
        words = binding.codes_words(n)
        g, u = rnd(n, dtype), rnd(n, dtype)
        hb, h = guarded(n, dtype, off)
        sb, s = guarded(n, dtype, off)
        cb, c = guarded(words, torch.int32)
        lmbp.reswiglu2_fwd(g, u, h=h, s=s, codes=c)
        for b, what in ((hb, "h"), (sb, "s")):
            check_guards(b, n, off, f"swiglu {what} n={n}")
        check_guards(cb, words, 0, f"swiglu codes n={n}")
        gb, dg = guarded(n, dtype, off)
        ub, du = guarded(n, dtype, off)
        lmbp.reswiglu2_bwd(rnd(n, dtype), u, s, c, dg=dg, du=du)
        check_guards(gb, n, off, f"swiglu dg n={n}")
        check_guards(ub, n, off, f"swiglu du n={n}")


@pytest.mark.parametrize("bits", [1, 2, 3, 4])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
def test_stepact_guards(bits, dtype):
    m = (1 << bits) - 1
    c = list(np.linspace(-3, 3, m))
    lv = list(np.linspace(0, 1, m + 1))
    per = 32 // bits
    for off in (0, 1):
        for n in ACT_SIZES:
            words = int(binding.lib().lmbp_stepact_codes_bytes(bits, n)) // 4
            yb, y = guarded(n, dtype, off)
            cb, cw = guarded(words, torch.int32)
            lmbp.stepact_fwd(rnd(n, dtype), "gelu", c, bits, y=y, codes=cw)
            check_guards(yb, n, off, f"stepact k={bits} y n={n}")
            check_guards(cb, words, 0, f"stepact k={bits} codes n={n}")
            used = bits * (n % per if n % per else per)
            if used < 32:
                last = int(cw[-1].item()) & 0xFFFFFFFF
                assert last >> used == 0, "unused code bits are not zero"
            db, dx = guarded(n, dtype, off)
            lmbp.stepact_bwd(rnd(n, dtype), cw, lv, bits, dx=dx)
            check_guards(db, n, off, f"stepact k={bits} dx n={n}")


NORM_SHAPES = [(1, 1), (3, 1000), (5, 1023), (7, 4096), (2, 8191), (4, 40000)]


@pytest.mark.parametrize("off", [0, 1])
@pytest.mark.parametrize("dtype", [torch.float32, torch.bfloat16])
@pytest.mark.parametrize("op", ["msln", "msrms"])
def test_norm_guards(op, dtype, off):
    fwd, bwd = getattr(lmbp, op + "_fwd"), getattr(lmbp, op + "_bwd")
    for rows, cols in NORM_SHAPES:
        n = rows * cols
        x = rnd(n, dtype).reshape(rows, cols)
        zb, z = guarded(n, dtype, off)
        rb, r = guarded(rows, torch.float32)
        fwd(x, 1e-5, z=z.view(rows, cols), rstd=r)
        check_guards(zb, n, off, f"{op} z {rows}x{cols}")
        check_guards(rb, rows, 0, f"{op} rstd {rows}x{cols}")
        db, dx = guarded(n, dtype, off)
        bwd(rnd(n, dtype).reshape(rows, cols), z.view(rows, cols), r, dx=dx.view(rows, cols))
        check_guards(db, n, off, f"{op} dx {rows}x{cols}")


LINEAR_SHAPES = [(1, 16, 24), (130, 272, 104), (257, 528, 64), (300, 400, 520)]


def test_linear_guards():
    for m, n, k in LINEAR_SHAPES:
        x = rnd(m * k, torch.bfloat16, 0.5).reshape(m, k)
        w = rnd(n * k, torch.bfloat16, 0.1).reshape(n, k)
        b = rnd(n, torch.bfloat16, 0.1)
        words = binding.codes_words(m * n)
        for act in ("gelu", "silu"):
            yb, y = guarded(m * n, torch.bfloat16)
            zb, z = guarded(m * n, torch.bfloat16)
            cb, c = guarded(words, torch.int32)
            lmbp.linear_act_fwd(x, w, b, act=act, y=y, codes=c, z=z)
            for buf, cnt, what in ((yb, m * n, "y"), (zb, m * n, "z"), (cb, words, "codes")):
                check_guards(buf, cnt, 0, f"linear {act} {what} {m}x{n}x{k}")
        wu = rnd(n * k, torch.bfloat16, 0.1).reshape(n, k)
        bufs = [guarded(m * n, torch.bfloat16) for _ in range(4)]
        cb, c = guarded(words, torch.int32)
        lmbp.linear_swiglu_fwd(x, w, wu, h=bufs[0][1], s=bufs[1][1], u=bufs[2][1], codes=c,
                               g=bufs[3][1])
        for (buf, _), what in zip(bufs, ("h", "s", "u", "g")):
            check_guards(buf, m * n, 0, f"swiglu linear {what} {m}x{n}x{k}")
        check_guards(cb, words, 0, f"swiglu linear codes {m}x{n}x{k}")
        # MS-RMSNorm in front: z [m, k] and rstd [m] as well
        zb, z = guarded(m * k, torch.bfloat16)
        rb, r = guarded(m, torch.float32)
        yb, y = guarded(m * n, torch.bfloat16)
        pb, pre = guarded(m * n, torch.bfloat16)
        cb, c = guarded(words, torch.int32)
        lmbp.msrms_linear_act_fwd(x, w, 1e-5, bias=b, act="silu", y=y, codes=c, z=z.view(m, k), rstd=r, pre=pre)
        for buf, cnt, what in ((yb, m * n, "y"), (pb, m * n, "pre"), (cb, words, "codes"), (zb, m * k, "z"),
                               (rb, m, "rstd")):
            check_guards(buf, cnt, 0, f"norm linear {what} {m}x{n}x{k}")
        bufs = [guarded(m * n, torch.bfloat16) for _ in range(4)]
        zb, z = guarded(m * k, torch.bfloat16)
        rb, r = guarded(m, torch.float32)
        cb, c = guarded(words, torch.int32)
        lmbp.msrms_linear_swiglu_fwd(x, w, wu, 1e-5, h=bufs[0][1], s=bufs[1][1], u=bufs[2][1], codes=c,
                                     g=bufs[3][1], z=z.view(m, k), rstd=r)
        for (buf, _), what in zip(bufs, ("h", "s", "u", "g")):
            check_guards(buf, m * n, 0, f"norm swiglu linear {what} {m}x{n}x{k}")
        check_guards(cb, words, 0, f"norm swiglu linear codes {m}x{n}x{k}")
        check_guards(zb, m * k, 0, f"norm swiglu linear z {m}x{n}x{k}")
        check_guards(rb, m, 0, f"norm swiglu linear rstd {m}x{n}x{k}")


def test_copy_guards():
    for nbytes in (16, 4096 + 5, 1 << 20):
        src = torch.randint(0, 255, (nbytes,), dtype=torch.uint8, device=DEV)
        buf = torch.full((nbytes + 2 * 64,), 0x5A, dtype=torch.uint8, device=DEV)
        dst = buf[64:64 + nbytes]
        lmbp.copy_bytes(src, dst)
        torch.cuda.synchronize()
        raw = buf.cpu().numpy()
        assert np.all(raw[:64] == 0x5A) and np.all(raw[64 + nbytes:] == 0x5A)
        assert np.array_equal(raw[64:64 + nbytes], src.cpu().numpy())
