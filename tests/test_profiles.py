"""The committed rocprofv3 summaries belong to the kernel code as it stands:
every profile names the code hash (comments and whitespace dropped) of the
sources its kernels are built from, and that hash must be the current one.
A change to a kernel's code therefore needs its profiles taken again; bench.py
stops reporting a traffic figure whose profile no longer matches."""
import glob
import json
import os
import re

import pytest

import bench

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PROFILES = os.path.join(ROOT, "profiles")

HASHES = {
    "decode": bench.kernel_source_hash(),
    "prefill": bench.kernel_source_hash(bench.PREFILL_SOURCES),
    "prefix": bench.kernel_source_hash(bench.PREFIX_SOURCES),
    "append": bench.kernel_source_hash(bench.APPEND_SOURCES),
}


def _md(name):
    with open(os.path.join(PROFILES, name), encoding="utf-8") as fh:
        return fh.read()


@pytest.mark.parametrize("path", sorted(glob.glob(os.path.join(PROFILES, "*.md"))),
                         ids=os.path.basename)
def test_every_profile_names_the_current_code(path):
    name = os.path.basename(path)
    text = _md(name)
    found = set(re.findall(r"\b[0-9a-f]{16}\b", text))
    if name.startswith("prefill"):
        need = {HASHES["prefill"]}
    else:
        need = {HASHES["decode"]}
        if name.startswith("grouped"):
            need.add(HASHES["prefix"])
        if name.startswith("append"):
            need.add(HASHES["append"])
    assert need <= found, f"{name}: names {sorted(found)}, current code {sorted(need)}"


@pytest.mark.parametrize("path", sorted(glob.glob(os.path.join(PROFILES, "*_traffic.json"))),
                         ids=os.path.basename)
def test_traffic_records_match_the_current_code(path):
    with open(path, encoding="utf-8") as fh:
        rec = json.load(fh)
    name = os.path.basename(path)
    want = HASHES["prefill"] if name.startswith("prefill") else HASHES["decode"]
    assert rec["kernel_source_hash"] == want
    if name.startswith("grouped"):
        assert rec["prefix_source_hash"] == HASHES["prefix"]
    # what bench.py would attach to its roofline record
    assert bench.load_traffic(want, path) == rec["hbm_bytes_per_launch"] > 0
