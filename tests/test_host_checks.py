"""Host-side checks of the C ABI, without a GPU: nova_kv_check_metadata
against a model of its rules written here, and the same checks built with
AddressSanitizer and UndefinedBehaviorSanitizer into a host program that
runs the argument checks and the metadata cases."""

import os
import shutil
import subprocess

import numpy as np
import pytest

import paper_2608_04074_amd as nk
from paper_2608_04074_amd import _native as nat

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OK, INVALID = nat.NOVA_KV_OK, nat.NOVA_KV_ERR_INVALID_ARG


def model(bs, bps, table, num_blocks, seq_lens, max_seq, start, n_new):
    """The metadata rules, written out: OK or INVALID."""
    cap = bs * bps
    if bs <= 0 or bps <= 0 or cap > 1 << 30 or n_new < 0:
        return INVALID
    batch = len(seq_lens) if seq_lens is not None else (len(start) if start is not None else 0)
    if seq_lens is not None and not 0 <= max_seq <= cap:
        return INVALID
    step = start is None and seq_lens is not None and n_new == 1
    if start is None and not step and n_new > 0:
        return INVALID

    def phys(b, blk):
        p = table[b * bps + blk] if table is not None else b * bps + blk
        if p < 0 or (num_blocks > 0 and p >= num_blocks):
            raise ValueError
        return p

    if seq_lens is not None and any(not 0 <= s <= max_seq for s in seq_lens):
        return INVALID
    rows, writers = set(), {}
    try:
        for b in range(batch):
            if start is not None:
                w = range(start[b], start[b] + n_new)
                if n_new > 0 and (start[b] < 0 or start[b] + n_new > cap):
                    return INVALID
            elif step and seq_lens[b] > 0:
                w = range(seq_lens[b] - 1, seq_lens[b])
            else:
                w = range(0)
            for t in w:
                p = phys(b, t // bs)
                if (p, t % bs) in rows:
                    return INVALID
                rows.add((p, t % bs))
                writers.setdefault(p, set()).add(b)
        if seq_lens is not None:
            for b in range(batch):
                for blk in range(-(-seq_lens[b] // bs)):
                    if writers.get(phys(b, blk), {b}) - {b}:
                        return INVALID
    except ValueError:
        return INVALID
    return OK


def random_case(rng):
    bs = int(rng.choice([1, 4, 16, 64]))
    bps = int(rng.integers(1, 9))
    batch = int(rng.integers(0, 6))
    cap = bs * bps
    num_blocks = int(rng.choice([0, batch * bps, batch * bps + 3, max(1, batch * bps - 2)]))
    table = None
    if rng.random() < 0.7:
        table = rng.permutation(max(batch * bps, 1) + 4)[: batch * bps].astype(np.int32)
        if rng.random() < 0.3 and table.size:
            table[rng.integers(table.size)] = int(rng.choice([-1, table[0], num_blocks, 10**6]))
    max_seq = int(rng.choice([cap, cap // 2, cap + 1, 0]))
    seq = None
    if rng.random() < 0.8:
        seq = rng.integers(0, max(cap, 1) + 1, size=batch).astype(np.int32)
        if rng.random() < 0.2 and batch:
            seq[rng.integers(batch)] = int(rng.choice([-3, cap + 5]))
    start, n_new = None, int(rng.choice([0, 1, 3]))
    if rng.random() < 0.4:
        start = rng.integers(-2, cap + 2, size=batch).astype(np.int32)
    return bs, bps, table, num_blocks, seq, max_seq, start, n_new


def cases(n, seed=0):
    rng = np.random.default_rng(seed)
    return [random_case(rng) for _ in range(n)]


def lib_status(bs, bps, table, num_blocks, seq, max_seq, start, n_new):
    try:
        nk.check_metadata(bs, bps, table, num_blocks, seq, max_seq, start, n_new)
        return OK
    except nat.NovaKVError as e:
        return e.status


def test_metadata_rules_by_example():
    table = np.array([[0, 1, 2, 3], [4, 5, 6, 7]], dtype=np.int32)
    ok = dict(block_size=16, blocks_per_seq=4, block_table=table, num_blocks=8, max_seq_len=64)
    nk.check_metadata(seq_lens=[64, 0], **ok)
    nk.check_metadata(seq_lens=[64, 0], n_new=1, **ok)            # the step skips the empty sequence
    nk.check_metadata(start_pos=[60, 0], n_new=4, **ok)
    bad = [
        (dict(seq_lens=[65, 1]), "seq_lens[0] = 65"),
        (dict(seq_lens=[-1, 1]), "seq_lens[0] = -1"),
        (dict(start_pos=[61, 0], n_new=4), "writes positions [61, 65)"),
        (dict(start_pos=[-1, 0], n_new=1), "writes positions [-1, 0)"),
        (dict(seq_lens=[1, 1], n_new=2), "writes need start_pos"),
    ]
    for kw, msg in bad:
        with pytest.raises(nat.NovaKVError, match=msg.replace("[", r"\[").replace("(", r"\(").replace(")", r"\)")):
            nk.check_metadata(**ok, **kw)
    with pytest.raises(nat.NovaKVError, match="physical block 9 outside"):
        nk.check_metadata(16, 4, np.array([[0, 1, 2, 9], [4, 5, 6, 7]]), 8, [64, 1], 64)
    with pytest.raises(nat.NovaKVError, match="write the same row"):
        nk.check_metadata(16, 4, np.array([[0, 1, 2, 3], [0, 5, 6, 7]]), 8, [1, 1], 64, n_new=1)
    with pytest.raises(nat.NovaKVError, match="reads physical block 3, which another sequence writes"):
        nk.check_metadata(16, 4, np.array([[0, 1, 2, 3], [3, 5, 6, 7]]), 8, [64, 10], 64, n_new=1)
    # an unknown pool size checks only that entries are >= 0
    nk.check_metadata(16, 4, np.array([[0, 1, 2, 90], [4, 5, 6, 7]]), 0, [64, 1], 64)


def test_metadata_check_follows_the_rules():
    for c in cases(3000):
        assert lib_status(*c) == model(*c), c


def _case_text(cs):
    out = [str(len(cs))]
    for bs, bps, table, nb, seq, max_seq, start, n_new in cs:
        batch = len(seq) if seq is not None else (len(start) if start is not None else 0)
        out.append(f"{bs} {bps} {int(table is not None)} {nb} {batch} {max_seq} {int(seq is not None)} "
                   f"{int(start is not None)} {n_new}")
        for x, n in ((table, batch * bps), (seq, batch), (start, batch)):
            if x is not None:
                out.append(" ".join(str(int(v)) for v in np.asarray(x).ravel()[:n]))
    return "\n".join(out) + "\n"


@pytest.mark.skipif(shutil.which("g++") is None, reason="g++ is not installed")
def test_host_checks_under_sanitizers(tmp_path):
    exe = tmp_path / "host_checks_asan"
    subprocess.run(["g++", "-std=c++17", "-O1", "-g", "-fno-omit-frame-pointer", "-fsanitize=address,undefined",
                    "-fno-sanitize-recover=all", "-I", os.path.join(ROOT, "include"),
                    os.path.join(ROOT, "paper_2608_04074_amd", "csrc", "host_checks.cpp"),
                    os.path.join(ROOT, "tests", "asan", "host_checks_driver.cpp"), "-o", str(exe)], check=True)
    cs = cases(2000, seed=1)
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=0:verify_asan_link_order=0",
               UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([str(exe)], input=_case_text(cs), capture_output=True, text=True, env=env, timeout=300)
    assert r.returncode == 0, r.stderr[-4000:]
    got = [int(x) for x in r.stdout.split()]
    assert got == [model(*c) for c in cs]
