"""The committed rocprofv3 summaries describe the committed kernels (CPU):
each names the hash of the sources it was taken on, the hash matches the
sources as they stand, and the HBM counters bench.py reads for the bench
line's `traffic` cover its pinned setting with plausible calibration."""
import hashlib
import importlib.util
import json
import os
import re

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PROFILES = os.path.join(ROOT, "profiles")
CSRC = os.path.join(ROOT, "paper_2608_16491_amd", "csrc")


def _bench():
    spec = importlib.util.spec_from_file_location("bench_mod", os.path.join(ROOT, "bench.py"))
    mod = importlib.util.module_from_spec(spec)
    spec.loader.exec_module(mod)
    return mod


def _sha(*names):
    h = hashlib.sha256()
    for n in names:
        with open(os.path.join(CSRC, n), "rb") as f:
            h.update(f.read())
    return h.hexdigest()[:16]


def _named_sha(md):
    text = open(os.path.join(PROFILES, md)).read()
    m = re.search(r"sha256\[:16\] = ([0-9a-f]{16})", text)
    assert m, md
    return m.group(1), text


def test_search_profiles_match_the_sources():
    b = _bench()
    sha = b.source_sha()
    for md in ("search_c2.md", "search_c2_mode0.md", "search_c2_fp16.md", "search_c2_sq.md"):
        named, text = _named_sha(md)
        assert named == sha, f"{md} was taken on other search sources"
        assert "rocprofv3" in text


def test_other_profiles_match_their_sources():
    named, _ = _named_sha("bruteforce_c2.md")
    assert named == _sha("bruteforce.hip", "exact.hip")
    named, _ = _named_sha("build_c2.md")
    assert named == _sha("build_gpu.hip")


def test_traffic_counters_cover_the_pinned_setting():
    b = _bench()
    tf = json.load(open(os.path.join(PROFILES, "search_c2_traffic.json")))
    assert tf["source_sha"] == b.source_sha()
    # a device copy of known size calibrates the counters: FETCH_SIZE reads
    # half the copied bytes on this setup, WRITE_SIZE all of them
    assert 1.5 < tf["fetch_factor"] < 2.5 and 0.8 < tf["write_factor"] < 1.2
    pinned = list(b.PINNED["c2"])
    ent = [e for e in tf["settings"] if [float(x) for x in e["setting"]] == [float(x) for x in pinned]]
    assert ent, "no counters at the pinned setting"
    for k in ("s_scan_kernel", "s_pool_kernel", "s_search_kernel"):
        kib = ent[0]["kernels"][k]
        assert kib["fetch_kib"] > 0 and kib["write_kib"] > 0
