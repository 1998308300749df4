"""Host-side checks of the C ABI that need no GPU: the library loads, exports
every symbol include/qevict.h declares, and rejects bad configurations before
touching the device."""
import os
import re

import pytest

import paper_2608_05326_amd as qv

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    src = open(os.path.join(ROOT, "include", "qevict.h")).read()
    return sorted(set(re.findall(r"\b(qevict_[a-z_]+)\s*\(", src)))


def test_library_exports_every_declared_symbol():
    lib = qv.load_library()
    names = _declared()
    assert len(names) >= 17
    for n in names:
        assert hasattr(lib, n), n
    assert set(names) == set(qv.SYMBOLS)


def _cfg(**kw):
    base = dict(batch=1, num_q_heads=32, num_kv_heads=8, window_tokens=32, quant_bits=4,
                max_context=32768 + 128, capacity_full=204, capacity_quant=307)
    base.update(kw)
    return qv.Config(**base)


def test_workspace_size_of_the_8b_32k_layer():
    n = qv.workspace_size(_cfg())
    # bf16 pool 204 x 8 heads x 16 KiB + quantized records 511 x 8 x 5 KiB + small state
    assert 204 * 8 * 16384 + 511 * 8 * 5120 < n < 60e6


@pytest.mark.parametrize("kw,status", [
    (dict(num_q_heads=30), qv.qevict.ERR_INVALID_ARG),
    (dict(head_dim=64), qv.qevict.ERR_UNSUPPORTED),
    (dict(window_tokens=48), qv.qevict.ERR_UNSUPPORTED),
    (dict(group_size=16), qv.qevict.ERR_UNSUPPORTED),
    (dict(quant_bits=3), qv.qevict.ERR_UNSUPPORTED),
    (dict(capacity_full=-1), qv.qevict.ERR_INVALID_ARG),
    (dict(capacity_full=3000, capacity_quant=2000), qv.qevict.ERR_UNSUPPORTED),
    (dict(num_q_heads=128, num_kv_heads=4), qv.qevict.ERR_UNSUPPORTED),
    (dict(retier_interval=0), qv.qevict.ERR_INVALID_ARG),
    (dict(flags=0x80), qv.qevict.ERR_INVALID_ARG),
    (dict(flags=qv.FLAG_ROUTING_QUEUE_WAIT), qv.qevict.ERR_INVALID_ARG),   # needs async routing
    (dict(flags=qv.FLAG_ROUTING_DEVICE_WAIT), qv.qevict.ERR_INVALID_ARG),
    (dict(flags=qv.FLAG_ASYNC_ROUTING | qv.FLAG_ROUTING_QUEUE_WAIT | qv.FLAG_ROUTING_DEVICE_WAIT),
     qv.qevict.ERR_INVALID_ARG),                                            # at most one order
    (dict(max_context=0), qv.qevict.ERR_INVALID_ARG),
    (dict(sink_tokens=65 * 32), qv.qevict.ERR_UNSUPPORTED),
    (dict(score_mode=4), qv.qevict.ERR_INVALID_ARG),
    (dict(rope_base=-1.0), qv.qevict.ERR_INVALID_ARG),
    (dict(rope_base=float("inf")), qv.qevict.ERR_INVALID_ARG),
    (dict(score_mode=qv.SCORE_PNORM, score_p=0.5), qv.qevict.ERR_INVALID_ARG),
    (dict(score_mode=qv.SCORE_PNORM, score_p=17.0), qv.qevict.ERR_INVALID_ARG),
    (dict(score_mode=qv.SCORE_DECAY, score_decay=0.0), qv.qevict.ERR_INVALID_ARG),
    (dict(score_mode=qv.SCORE_DECAY, score_decay=1.5), qv.qevict.ERR_INVALID_ARG),
])
def test_bad_configs_are_rejected(kw, status):
    with pytest.raises(qv.QEvictError) as e:
        qv.workspace_size(_cfg(**kw))
    assert e.value.status == status


def test_ranking_modes_are_accepted():
    base = qv.workspace_size(_cfg())
    assert qv.workspace_size(_cfg(score_mode=qv.SCORE_DECAY, score_decay=0.99)) == base
    # key-norm mode stages the prompt windows' scores ([B][n_w] fp32) after the units
    kn = qv.workspace_size(_cfg(score_mode=qv.SCORE_KEY_NORM))
    assert base + 4 * 1028 <= kn <= base + 4 * 1028 + 256
    # RoPE: a float32 (cos, sin) table of max_context x 64 pairs after the units
    rp = qv.workspace_size(_cfg(rope_base=10000.0))
    assert rp == base + 8 * (32768 + 128) * 64
    # p-norm mode: the same staging plus {completed-period sum, running u} per window and unit
    pn = qv.workspace_size(_cfg(score_mode=qv.SCORE_PNORM, score_p=3.0))
    n_units = 1 * 1
    assert kn + n_units * 8 * 1028 <= pn <= kn + n_units * (8 * 1028 + 256)


def test_status_strings():
    lib = qv.load_library()
    assert lib.qevict_status_string(0) == b"ok"
    assert lib.qevict_status_string(-6) == b"capacity exceeded"


def test_prefill_scores_scratch_size():
    cfg = _cfg()
    # per (sequence, KV head): a (max, sum) pair per row and 64-key chunk, a sum per
    # row and window, (M, 1/L) per row
    rows, n_chunks, n_w = 4 * 32, 32768 // 64, 32768 // 32
    n = qv.qevict.prefill_scores_scratch_size(cfg, 32768, 32)
    expect = 8 * (8 * rows * n_chunks) + 4 * (8 * rows * n_w) + 8 * (8 * rows)
    assert expect <= n <= expect + 3 * 256
    for T, n_obs in [(0, 1), (100, 0), (100, 101), (10 ** 6, 1), (8192, 4097)]:
        with pytest.raises(qv.QEvictError) as e:
            qv.qevict.prefill_scores_scratch_size(cfg, T, n_obs)
        assert e.value.status == qv.qevict.ERR_INVALID_ARG


def test_c_program_uses_the_abi(tmp_path):
    """tests/c/abi_host.c: the header compiles as C99 and the host-only calls
    work from C, linked against the built library."""
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no C compiler")
    here = os.path.dirname(os.path.abspath(__file__))
    root = os.path.dirname(here)
    lib_dir = os.path.join(root, "paper_2608_05326_amd")
    exe = str(tmp_path / "abi_host")
    subprocess.run([gcc, "-std=c99", "-Wall", "-Werror", "-I", os.path.join(root, "include"),
                    os.path.join(here, "c", "abi_host.c"), "-L", lib_dir, "-lqevict",
                    "-Wl,-rpath," + lib_dir, "-o", exe], check=True)
    r = subprocess.run([exe], capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "FAIL" not in r.stdout
