"""C-ABI boundary checks that need no GPU: the library loads, exports every symbol
include/libbpt.h declares, validates arguments and sizes its buffers linearly in S."""
import ctypes
import os
import re

import pytest

from paper_2305_19370_amd import bpt

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "libbpt.h")

pytestmark = pytest.mark.skipif(not os.path.exists(bpt.LIB_PATH), reason="libbpt.so not built")


def declared_symbols():
    txt = open(HEADER).read()
    txt = re.sub(r"/\*.*?\*/", "", txt, flags=re.S)
    return sorted(set(re.findall(r"\b(bpt_[a-z_]+)\s*\(", txt)))


def test_exports_match_header():
    lib = bpt.load()
    decl = declared_symbols()
    assert decl, "no declarations parsed"
    for name in decl:
        assert hasattr(lib, name), f"{name} declared in libbpt.h but not exported"
    assert set(decl) == set(bpt.EXPORTS)


def cfg(**kw):
    base = dict(B=1, S=512, D=256, H=4, F=1024, Bq=128, Bkv=128, causal=True, dtype="f32")
    base.update(kw)
    return bpt.make_config(**base)


def test_valid_configs():
    assert bpt.validate(cfg()) == 0
    assert bpt.validate(cfg(D=4096, H=32, F=16384, S=32768, Bq=1024, Bkv=1024, dtype="bf16")) == 0
    assert bpt.validate(cfg(S=250, Bq=1, Bkv=250)) == 0          # ragged, extreme blocks
    assert bpt.validate(cfg(B=4, S=96000, D=1024, H=8, F=4096, Bq=1024, Bkv=1024, dtype="bf16")) == 0


@pytest.mark.parametrize("kw,code", [
    (dict(D=250, H=5), 2),             # dh = 50 unsupported
    (dict(D=256, H=3), 1),             # D % H != 0
    (dict(D=320, H=5), 2),             # dh = 64 but D not a multiple of 64? (320 = 5*64 is fine) -> see below
    (dict(F=1000), 2),                 # F % 64
    (dict(Bq=0), 1), (dict(Bq=513), 1), (dict(Bkv=0), 1), (dict(Bkv=600), 1),
    (dict(B=0), 1), (dict(S=0), 1), (dict(H=0), 1),
    (dict(D=512, H=2), 2),             # dh = 256
])
def test_invalid_configs(kw, code):
    c = cfg(**kw)
    if kw == dict(D=320, H=5):
        assert bpt.validate(c) == 0     # 320 = 5 x 64 is a supported shape
        return
    assert bpt.validate(c) == code
    assert bpt.saved_bytes(c) == 0 and bpt.workspace_bytes(c, False) == 0 and bpt.workspace_bytes(c, True) == 0
    assert bpt.group_rows(c) == -1
    assert bpt.load().bpt_last_error().decode()


def test_bad_enums_and_eps():
    c = cfg()
    c.dtype = 7
    assert bpt.validate(c) == 1
    c = cfg()
    c.causal = 2
    assert bpt.validate(c) == 1
    c = cfg()
    c.ln_eps = 0.0
    assert bpt.validate(c) == 1
    c = cfg()
    c.group_blocks = -1
    assert bpt.validate(c) == 1
    assert bpt.load().bpt_validate(None) == 1


def test_calls_reject_bad_pointers_before_launch():
    """Null / aliased / misaligned pointers and short workspaces fail on the host; nothing launches."""
    lib = bpt.load()
    c = cfg()
    p = bpt.Params(*([64 * 1024] * 12))
    ws = bpt.workspace_bytes(c, False)
    # NULL X
    assert lib.bpt_layer_fwd(ctypes.byref(c), None, ctypes.byref(p), 4096, 8192, 1 << 20, ws, None) == 1
    # Y aliases X
    assert lib.bpt_layer_fwd(ctypes.byref(c), 4096, ctypes.byref(p), 4096, 8192, 1 << 20, ws, None) == 1
    # misaligned Y
    assert lib.bpt_layer_fwd(ctypes.byref(c), 4096, ctypes.byref(p), 4100, 8192, 1 << 20, ws, None) == 1
    # short workspace
    assert lib.bpt_layer_fwd(ctypes.byref(c), 4096, ctypes.byref(p), 8192, 16384, 1 << 20, ws - 1, None) == 3
    assert "workspace" in lib.bpt_last_error().decode()
    # NULL weight
    p0 = bpt.Params(*([64 * 1024] * 12))
    p0.W1 = None
    assert lib.bpt_layer_fwd(ctypes.byref(c), 4096, ctypes.byref(p0), 8192, 16384, 1 << 20, ws, None) == 1
    g = bpt.Grads()
    wsb = bpt.workspace_bytes(c, True)
    assert lib.bpt_layer_bwd(ctypes.byref(c), 4096, ctypes.byref(p), 8192, 12288, 12288, ctypes.byref(g),
                             1 << 20, wsb, None) == 1      # dX aliases dY
    assert lib.bpt_layer_bwd(ctypes.byref(c), 4096, ctypes.byref(p), 8192, 12288, 16384, ctypes.byref(g),
                             1 << 20, wsb - 256, None) == 3
    bad = bpt.make_config(1, 512, 250, 5, 1024, 128, 128, True, "f32")
    assert lib.bpt_layer_fwd(ctypes.byref(bad), 4096, ctypes.byref(p), 8192, 16384, 1 << 20, ws, None) == 2


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_sizes_linear_in_S(dtype):
    """Saved and workspace bytes have no S^2 or S*F term: second differences in S vanish
    (up to 64-token padding and 256-byte alignment)."""
    D, H, F, Bq = 1024, 8, 4096, 256
    Ss = [8192, 16384, 24576, 32768]     # multiples of 64 and of the group rows

    def conf(S):
        c = bpt.make_config(1, S, D, H, F, Bq, Bq, True, dtype)
        c.group_blocks = 8192 // Bq         # groups of 8192 rows, fewer than S
        return c
    for fn in (lambda c: bpt.saved_bytes(c), lambda c: bpt.workspace_bytes(c, False),
               lambda c: bpt.workspace_bytes(c, True)):
        v = [fn(conf(S)) for S in Ss]
        d1 = [b - a for a, b in zip(v, v[1:])]
        assert max(d1) - min(d1) <= 4096, (v, d1)
        per_token = d1[0] / 8192
        assert per_token < 200 * D, per_token           # O(D) bytes per token, never O(F) or O(S)
    sp = bpt.saved_bytes(bpt.make_config(1, 8192, D, H, F, Bq, Bq, True, dtype))
    es = 2 if dtype == "bf16" else 4
    assert sp >= 8192 * D * (4 * es + 4)                # Q, K, V, O, h at least


def test_group_rows_and_describe():
    c = bpt.make_config(1, 32768, 4096, 32, 16384, 1024, 1024, True, "bf16")
    assert bpt.group_rows(c) == 16384                   # automatic: 16384 rows at F >= 8192
    for F, rows in ((2048, 65536), (4096, 32768), (8192, 16384), (20480, 16384)):   # else 2^27 / F
        assert bpt.group_rows(bpt.make_config(1, 65536, 1024, 8, F, 1024, 1024, True, "bf16")) == rows
    assert bpt.group_rows(bpt.make_config(1, 65536, 1024, 8, 4096, 1000, 1000, True, "bf16")) == 33000
    c.group_blocks = 1
    assert bpt.group_rows(c) == 1024
    c.group_blocks = 100
    assert bpt.group_rows(c) == 32768
    c2 = cfg(S=250, Bq=100)
    c2.group_blocks = 2
    assert bpt.group_rows(c2) == 200
    txt = bpt.describe(c)
    assert "group rows=32768" in txt and "MFMA" in txt
    # the workspace holds one group's [rows, F] intermediate, not the sequence's
    c.group_blocks = 1
    small = bpt.workspace_bytes(c, False)
    c.group_blocks = 8
    big = bpt.workspace_bytes(c, False)
    assert big - small >= 7 * 1024 * 16384 * 2


def test_groups_of_whole_sequences():
    """A group holds several whole sequences when at least two fit in group_blocks * Bq
    rows (and never more sequences than the batch has); otherwise a run of one."""
    c = bpt.make_config(2, 4096, 2048, 16, 16384, 512, 512, True, "bf16")     # 8192 rows: both sequences
    assert bpt.group_rows(c) == 8192 and "2 sequence(s) x 4096 rows" in bpt.describe(c)
    c = bpt.make_config(5, 2048, 2048, 16, 16384, 1024, 1024, True, "bf16")    # 16384 rows: all 5
    assert bpt.group_rows(c) == 5 * 2048
    c = bpt.make_config(5, 2048, 2048, 16, 16384, 1024, 1024, True, "bf16")
    c.group_blocks = 8                                                          # 8192 rows: 4 of 5 fit
    assert bpt.group_rows(c) == 4 * 2048
    c = bpt.make_config(5, 2048, 2048, 16, 8192, 1024, 1024, True, "bf16")     # 16384 rows at F = 8192
    assert bpt.group_rows(c) == 5 * 2048
    c = bpt.make_config(3, 9000, 2048, 16, 16384, 1000, 1000, True, "bf16")    # only one fits: a run
    assert bpt.group_rows(c) == 9000 and "1 sequence(s) x 9000 rows" in bpt.describe(c)
    c = bpt.make_config(1, 100, 256, 2, 512, 10, 10, True, "bf16")             # B = 1
    assert bpt.group_rows(c) == 100
    c = bpt.make_config(4, 100, 256, 2, 512, 10, 10, True, "bf16")
    c.group_blocks = 25                                                         # 250 rows: 2 sequences
    assert bpt.group_rows(c) == 200


def test_saved_layout_offsets():
    for dtype in ("f32", "bf16"):
        c = cfg(B=2, S=250, dtype=dtype)
        lay = bpt.saved_layout(c)
        offs = [lay[k] for k in bpt.SAVED_FIELDS[:-1]]
        assert offs == sorted(offs) and all(o % 256 == 0 for o in offs)
        assert lay["total"] == bpt.saved_bytes(c)
        es = 2 if dtype == "bf16" else 4
        T, D, Sp = 500, 256, 256
        assert lay["o"] - lay["qkv"] >= T * 3 * D * es
        assert lay["h"] - lay["lse"] >= 2 * 4 * Sp * 4


def test_status_strings():
    lib = bpt.load()
    assert lib.bpt_status_string(0) == b"BPT_OK"
    assert lib.bpt_status_string(3) == b"BPT_ERR_WORKSPACE"
    assert lib.bpt_status_string(99) == b"BPT_ERR_UNKNOWN"


def test_activation_is_validated():
    cfg = bpt.make_config(1, 256, 256, 2, 512, 64, 64, True, "bf16", activation="relu")
    assert bpt.validate(cfg) == 0 and "relu" in bpt.describe(cfg)
    cfg.activation = 7
    assert bpt.validate(cfg) == 1


def test_dropout_is_validated_and_sizes_its_workspace():
    """A rate outside [0, 1) is rejected; a rate > 0 adds the fp32 FFN-output block
    (forward) and the masked dY (backward) to the workspaces."""
    base = bpt.make_config(1, 256, 256, 2, 512, 64, 64, True, "bf16")
    drop = bpt.make_config(1, 256, 256, 2, 512, 64, 64, True, "bf16", dropout=0.1, dropout_seed=2 ** 64 - 1)
    assert bpt.validate(drop) == 0
    assert bpt.workspace_bytes(drop, False) > bpt.workspace_bytes(base, False)
    assert bpt.workspace_bytes(drop, True) >= bpt.workspace_bytes(base, True) + 256 * 256 * 2
    for bad in (1.0, -0.1, float("nan")):
        drop.dropout = bad
        assert bpt.validate(drop) == 1


def test_gpt_step_entries_validate_before_launch():
    """Embedding, final LayerNorm and AdamW reject bad configurations and pointers
    on the host (fake, never-dereferenced addresses; nothing launches)."""
    lib = bpt.load()
    e = bpt.make_embed_config(2, 64, 256, 1000, dtype="bf16")
    assert lib.bpt_embed_fwd(ctypes.byref(e), None, 4096, None, 8192, None) == 1          # NULL tokens
    assert lib.bpt_embed_fwd(ctypes.byref(e), 4096, 4104, None, 8192, None) == 1          # misaligned Wte
    bad = bpt.make_embed_config(2, 64, 252, 1000)                                           # D % 8
    assert lib.bpt_embed_fwd(ctypes.byref(bad), 4096, 8192, None, 16384, None) == 2
    bad = bpt.EmbedConfig(2, 64, 256, 1000, 7, 0)                                           # dtype
    assert lib.bpt_embed_bwd(ctypes.byref(bad), 4096, 8192, 16384, None, None) == 1
    assert lib.bpt_embed_bwd(ctypes.byref(e), 4096, None, 16384, None, None) == 1         # NULL dX

    ln = bpt.make_ln_config(128, 256, 1e-5, in_dtype="bf16")
    n = bpt.ln_workspace_bytes(ln)
    assert n >= 2 * 256 * 4 + 128 * 256 * 4          # partials + fp32 copy of a bf16 dY
    assert bpt.ln_workspace_bytes(bpt.make_ln_config(128, 256, 1e-5, in_dtype="f32")) < n
    assert bpt.ln_workspace_bytes(bpt.make_ln_config(0, 256)) == 0
    assert bpt.ln_workspace_bytes(bpt.LnConfig(128, 256, -1.0, 0, 0, 0)) == 0
    assert lib.bpt_ln_fwd(ctypes.byref(ln), 4096, None, None, 4096, 8192, 12288, None) == 1   # Y aliases X
    assert lib.bpt_ln_bwd(ctypes.byref(ln), 4096, None, 8192, 12288, 16384, 20480, 24576, None,
                          1 << 20, n, None) == 1                                            # dg without db
    assert lib.bpt_ln_bwd(ctypes.byref(ln), 4096, None, 8192, 12288, 16384, 20480, None, None,
                          1 << 20, n - 1, None) == 3                                        # short workspace

    a = bpt.AdamWConfig(1e-3, 0.9, 0.95, 1e-8, 0.1, 1, 1)
    assert lib.bpt_adamw_step(ctypes.byref(a), 0, None, None, None, None, None, None) == 0    # empty: no-op
    assert lib.bpt_adamw_step(ctypes.byref(a), 8, None, 4096, 8192, 12288, None, None) == 1   # NULL p
    assert lib.bpt_adamw_step(ctypes.byref(a), 8, 4100, 4096, 8192, 12288, None, None) == 1   # misaligned
    for bad in (bpt.AdamWConfig(1e-3, 1.0, 0.95, 1e-8, 0.1, 1, 1), bpt.AdamWConfig(1e-3, 0.9, 0.95, 0.0, 0.1, 1, 1),
                bpt.AdamWConfig(1e-3, 0.9, 0.95, 1e-8, 0.1, 1, 0), bpt.AdamWConfig(-1.0, 0.9, 0.95, 1e-8, 0.1, 1, 1)):
        assert lib.bpt_adamw_step(ctypes.byref(bad), 8, 4096, 8192, 12288, 16384, None, None) == 1


def test_probe_library_exports_match_header():
    """libbpt_probe.so (the matrix-core ceiling probe bench.py --mfma-probe times) exports
    what include/bpt_probe.h declares, and rejects invalid arguments without launching."""
    path = os.path.join(os.path.dirname(bpt.LIB_PATH), "libbpt_probe.so")
    if not os.path.exists(path):
        pytest.skip("libbpt_probe.so not built")
    txt = re.sub(r"/\*.*?\*/", "", open(os.path.join(ROOT, "include", "bpt_probe.h")).read(), flags=re.S)
    decl = sorted(set(re.findall(r"\b(bpt_[a-z_]+)\s*\(", txt)))
    assert decl == ["bpt_probe_mfma_loop"]
    lib = ctypes.CDLL(path)
    fn = lib.bpt_probe_mfma_loop
    fn.restype = ctypes.c_int32
    fn.argtypes = [ctypes.c_int64, ctypes.c_int32, ctypes.c_int32, ctypes.c_void_p, ctypes.c_void_p,
                   ctypes.c_void_p]
    assert fn(0, 10, 0, 4096, 4096, None) == 1          # no workgroups
    assert fn(1 << 25, 10, 0, 4096, 4096, None) == 1    # too many
    assert fn(8, 0, 0, 4096, 4096, None) == 1           # no iterations
    assert fn(8, 10, 0, None, 4096, None) == 1          # null seed
    assert fn(8, 10, 1, 4096, None, None) == 1          # null out
    assert fn(8, 10, 8, 4096, 4096, None) == 1          # no such mode
    assert fn(8, 10, -1, 4096, 4096, None) == 1         # no such mode
