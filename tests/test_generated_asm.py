"""The inline-assembly MFMA phase of the ping-pong attention kernel is
generated text: the committed include must equal what its generator
writes, and the generator's fragment schedule must keep its invariants."""
import importlib.util
import os
import re
import subprocess
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
CSRC = os.path.join(ROOT, "paper_2608_26112_amd", "csrc")


def _gen():
    spec = importlib.util.spec_from_file_location("gen_mfma_phase",
                                                  os.path.join(CSRC, "gen_mfma_phase.py"))
    m = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(m)
    return m


def test_include_matches_generator():
    out = subprocess.run([sys.executable, os.path.join(CSRC, "gen_mfma_phase.py")],
                         capture_output=True, text=True, check=True).stdout
    with open(os.path.join(CSRC, "mfma_phase_d128.inc")) as f:
        assert f.read() == out


def _simulate(lines):
    """Replays one statement: LDS reads complete in order; returns the
    ring slot contents each MFMA reads (fragment ids) and checks that every
    read's slot is not refilled before its MFMA issued."""
    pending, ready, reads_issued = [], {}, 0
    slot_of_read = []
    mfmas = []
    for ln in lines:
        m = re.match(r"ds_read_\w+ v\[(\d+):(\d+)\]", ln)
        if m:
            pending.append((int(m.group(1)), int(m.group(2)), reads_issued))
            reads_issued += 1
            continue
        m = re.match(r"s_waitcnt lgkmcnt\((\d+)\)", ln)
        if m:
            keep = int(m.group(1))
            while len(pending) > keep:
                lo, hi, rid = pending.pop(0)
                for r in range(lo, hi + 1):
                    ready[r] = rid
            continue
        m = re.match(r"v_mfma_f32_32x32x16_bf16 \S+, v\[(\d+):(\d+)\]", ln)
        if m:
            lo, hi = int(m.group(1)), int(m.group(2))
            # every register of the A operand has landed and is not being refilled
            assert all(r in ready for r in range(lo, hi + 1)), ln
            assert not any(plo <= hi and phi >= lo for plo, phi, _ in pending), ln
            mfmas.append(tuple(ready[r] for r in range(lo, hi + 1)))
    assert not pending
    return mfmas


def test_fragment_schedule():
    g = _gen()
    for pv, qk, n in ((True, True, 32), (True, False, 16), (False, True, 16)):
        lines = g.body(pv, qk)
        assert lines[0].startswith("s_nop") and lines[-1].startswith("s_nop")
        mf = _simulate(lines)
        assert len(mf) == n
        # the MFMAs read the fragments in order: PV reads two per fragment
        # (its two transposed halves), QK^T one
        per = [2] * (16 if pv else 0) + [1] * (16 if qk else 0)
        first = 0
        for k, regs in enumerate(mf):
            assert set(regs) == set(range(first, first + per[k])), (k, regs)
            first += per[k]
