"""The parity record writer and its summary (host logic, no GPU)."""
import json

import parity_log


def test_record_and_summary(tmp_path, monkeypatch):
    path = tmp_path / "rec.jsonl"
    monkeypatch.setenv("DERF_PARITY_RECORD", str(path))
    np = __import__("numpy")
    parity_log.record(test="a", kind="cells", samples=np.int64(100), near_bisector=3,
                      mismatches=0)
    parity_log.record(test="b", kind="pixels", rays=7, max_abs_rgb=np.float32(1.5e-7),
                      max_abs_depth=2e-7, max_abs_opacity=3e-8, tol=1e-4)
    parity_log.record(test="c", kind="other", x=np.arange(2))
    recs = [json.loads(line) for line in open(path)]
    assert recs[0]["samples"] == 100 and recs[2]["x"] == [0, 1]
    text = parity_log.summarize(str(path))
    assert "### cells" in text and "| a | 100 | 3 | 0 |" in text
    assert "### pixels" in text and "| b | 7 | 1.5e-07 |" in text
    assert "### other" in text and "| c | [0, 1] |" in text


def test_no_record_without_the_variable(tmp_path, monkeypatch):
    monkeypatch.delenv("DERF_PARITY_RECORD", raising=False)
    parity_log.record(test="a", kind="cells")
    assert not list(tmp_path.iterdir())
