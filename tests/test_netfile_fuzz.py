"""Robustness of the host-side parsing and planning (CPU, no GPU needed).

Seeded mutations of the shipped NetFiles (byte flips, inserted keywords and
extreme numbers, cuts, long runs) go through cnn_netfile_parse; every text
must come back as a layer list or as an error status, never a crash, and a
parsed list (with random fields then set to extreme values) goes through the
shape and workspace planners, which must also answer with a status.  The
same driver was run under host AddressSanitizer and UndefinedBehaviorSanitizer
builds of the library with many more iterations.
"""
import ctypes
import os
import random

from paper_1511_07376_amd import cnn

TOKENS = [b"conv", b"fc", b"pool", b"lrn", b"relu", b"softmax", b"input", b"max", b"avg", b"out=", b"in=",
          b"kernel=", b"stride=", b"pad=", b"groups=", b"size=", b"alpha=", b"=", b"#", b"\n", b" ", b"-1",
          b"0", b"2147483647", b"99999999999", b"1e30", b"nan", b"3x", b"execution_mode", b"graph",
          b"sequential", b"auto_tuning", b"on", b"off", b"ceil", b"\t", b"\xff"]
FIELDS = ["out_channels", "kernel_h", "stride_w", "pad_h", "groups", "lrn_size", "in_features", "type"]
EXTREMES = [-5, 0, 1, 3, 7, 1 << 20, 2147483647]


def _mutate(rng, s: bytearray) -> bytes:
    for _ in range(rng.randint(1, 8)):
        op = rng.random()
        pos = rng.randint(0, max(0, len(s) - 1))
        if op < 0.3 and s:
            s[pos] = rng.randint(1, 255)
        elif op < 0.55:
            s[pos:pos] = rng.choice(TOKENS)
        elif op < 0.75 and s:
            del s[pos:pos + rng.randint(1, 40)]
        elif op < 0.85:
            s = s[:pos]
        else:
            s[pos:pos] = b"x" * rng.randint(1, 3000)
    return bytes(s)


def test_mutated_netfiles_parse_or_fail_cleanly():
    seeds = [open(os.path.join(cnn.NETFILE_DIR, f), "rb").read() for f in sorted(os.listdir(cnn.NETFILE_DIR))]
    rng = random.Random(11)
    parsed = 0
    for _ in range(3000):
        text = _mutate(rng, bytearray(rng.choice(seeds)))
        n, cfg = ctypes.c_int(), cnn.cnn_netfile_config()
        rc = cnn.lib.cnn_netfile_parse(text, None, 0, ctypes.byref(n), ctypes.byref(cfg))
        assert rc in (cnn.CNN_OK, cnn.CNN_ERR_INVALID, cnn.CNN_ERR_UNSUPPORTED), rc
        if rc != cnn.CNN_OK:
            assert cnn.cnn_last_error()
            continue
        parsed += 1
        cap = rng.choice([0, max(n.value - 1, 0), n.value])
        descs = (cnn.cnn_layer_desc * max(cap, 1))()
        m = ctypes.c_int()
        rc = cnn.lib.cnn_netfile_parse(text, descs, cap, ctypes.byref(m), ctypes.byref(cfg))
        if cap < n.value:
            assert rc != cnn.CNN_OK      # the caller's array is too small
            continue
        assert rc == cnn.CNN_OK and m.value == n.value
        oc, oh, ow = ctypes.c_int(), ctypes.c_int(), ctypes.c_int()
        for _ in range(3):
            if m.value:
                setattr(descs[rng.randrange(m.value)], rng.choice(FIELDS), rng.choice(EXTREMES))
            N = rng.choice([0, 1, 64])
            rc = cnn.lib.cnn_net_out_shape(descs, m.value, N, cfg.in_channels, cfg.in_height, cfg.in_width,
                                           ctypes.byref(oc), ctypes.byref(oh), ctypes.byref(ow))
            assert rc in (cnn.CNN_OK, cnn.CNN_ERR_INVALID, cnn.CNN_ERR_UNSUPPORTED), rc
            cnn.lib.cnn_net_workspace_bytes(descs, m.value, N, cfg.in_channels, cfg.in_height, cfg.in_width)
    assert parsed > 100
