"""The CPU model of the inter-workgroup protocols (tests/protocol_model.cpp).

The model runs the tile-ticket, epoch-tagged status-word, decoupled look-back
(Section 2.1), epoch-wrap and per-row arrival rules of the kernels with one
std::thread per workgroup, fewer resident slots than workgroups and
workgroups started out of order, then checks every result against the serial
scan, the error flag and the workspace invariant after every launch.  It
shows on a machine without a GPU that a protocol change neither deadlocks nor
reads a stale word.  Each planted protocol mistake must be caught, the
correct protocol must pass on many seeds and under ThreadSanitizer, and the
per-XCD ticket scheme (tile = 8 * per-XCD ticket + XCD) must stall under a
legal dispatch that holds one XCD back, where the single ticket does not.
"""
import os
import shutil
import subprocess

import pytest

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "protocol_model.cpp")
pytestmark = pytest.mark.skipif(shutil.which("g++") is None, reason="g++ is needed")

MUTATIONS = ["blockidx_tiles", "no_ticket_reset", "ignore_epoch", "no_wrap_clear", "x_as_zero",
             "drop_p_lane", "window_from_self", "row_plain_count", "row_no_clear_counter",
             "xcd_tickets", "persistent_reset_at_tiles"]


def _build(out, *flags):
    subprocess.run(["g++", "-std=c++17", "-pthread", "-Wall", "-Wextra", "-Werror", *flags, "-o",
                    str(out), SRC], check=True, capture_output=True)
    return str(out)


@pytest.fixture(scope="module")
def model(tmp_path_factory):
    return _build(tmp_path_factory.mktemp("model") / "protocol_model", "-O2")


def _run(exe, *args, timeout=120):
    return subprocess.run([exe, *args], capture_output=True, text=True, timeout=timeout)


def test_mutation_list_matches(model):
    listed = _run(model, "--list-mutations").stdout.split()
    assert listed == ["none"] + MUTATIONS


@pytest.mark.parametrize("seed", range(1, 13))
def test_protocol_holds(model, seed):
    r = _run(model, "--seed", str(seed))
    assert r.returncode == 0 and "MODEL_OK" in r.stdout, r.stderr[-2000:]


@pytest.mark.parametrize("mutation", MUTATIONS)
def test_planted_mistake_is_caught(model, mutation):
    for seed in (1, 2, 3):
        r = _run(model, "--mutation", mutation, "--seed", str(seed))
        assert r.returncode == 1 and "FAIL:" in r.stderr, (mutation, seed, r.stdout, r.stderr)


def test_held_xcd_dispatch(model):
    """Blocks dispatched in order except one XCD's, which come last: the
    single ticket counter hands tiles out in arrival order and finishes; one
    counter per XCD leaves the resident workgroups waiting on tiles that no
    running workgroup holds (the model's bounded wait reports it)."""
    ok = _run(model, "--scenario", "held_xcd")
    assert ok.returncode == 0 and "ok held_xcd" in ok.stdout, ok.stderr
    bad = _run(model, "--scenario", "held_xcd", "--mutation", "xcd_tickets")
    assert bad.returncode == 1 and "error flag set" in bad.stderr, bad.stderr


def test_under_thread_sanitizer(tmp_path):
    """Every shared word of the model is an atomic: ThreadSanitizer finds no
    data race in the correct protocol."""
    if not subprocess.run(["gcc", "-print-file-name=libtsan.so"], capture_output=True,
                          text=True).stdout.strip().startswith("/"):
        pytest.skip("no ThreadSanitizer runtime")
    exe = _build(tmp_path / "protocol_model_tsan", "-O1", "-g", "-fsanitize=thread")
    env = dict(os.environ, TSAN_OPTIONS="halt_on_error=1:exitcode=66")
    for seed in (1, 2):
        r = subprocess.run([exe, "--quick", "--seed", str(seed)], capture_output=True, text=True,
                           timeout=600, env=env)
        assert r.returncode == 0 and "ThreadSanitizer" not in r.stderr, r.stderr[-3000:]
