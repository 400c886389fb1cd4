"""The phase-clock diagnostic finds every anchor in the current on-chip
kernel source (it instruments a copy by text insertion)."""
import os

from paper_2607_06763_amd import phase_clocks as P

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def test_instrumentation_anchors_match_the_kernel():
    with open(os.path.join(ROOT, "paper_2607_06763_amd", "csrc", "gdn_verify.hip")) as f:
        src = f.read()
    out = P._instrument(src)
    stamps = [ln.strip() for ln in out.splitlines() if ln.strip().startswith("TS(")]
    assert len(stamps) == 11          # prologue 2, per head 8, end 1
    assert out.count("TR(6") == 2      # real-time counter at the start and the end
    assert "TS(40);" in stamps
    assert "unsigned long long* stamps;" in out and 'extern "C" void gdn_phase_stamps' in out
    # every phase boundary the summary reads is stamped
    for _, a, b in P.PHASES:
        for k in (a, b):
            assert any(s.startswith(f"TS({k}") for s in stamps), k


def test_chunked_instrumentation_anchors_match_the_kernel():
    with open(os.path.join(ROOT, "paper_2607_06763_amd", "csrc", "gdn_chunked.hip")) as f:
        out = P._instrument_chunked(f.read())
    stamps = [ln.strip() for ln in out.splitlines() if ln.strip().startswith("TS(")]
    assert len(stamps) == 8           # metadata, phase A, phase B, 4 per block, end
    assert "TS(127);" in stamps and 'extern "C" void gdn_chunk_stamps' in out
