"""The rocprofv3 summaries under profiles/ describe the kernels as they are:
each states the sha256 (first 16 hex digits) of the sources its kernels are
built from, and that hash must match the sources in the tree. A kernel
change without a new profile fails here."""
import hashlib
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
PROFILES = os.path.join(ROOT, "profiles")
PKG = os.path.join(ROOT, "paper_2607_07046_amd")
LINE = re.compile(r"source hash \(sha256 of ([^,]+), first 16 hex\): `([0-9a-f]{16})`")


def _profiles():
    return sorted(f for f in os.listdir(PROFILES) if f.endswith(".md"))


@pytest.mark.parametrize("name", _profiles())
def test_profile_hash_matches_sources(name):
    text = open(os.path.join(PROFILES, name)).read()
    m = LINE.search(text)
    assert m, f"{name} states no source hash"
    files = [f.strip() for f in m.group(1).split("+")]
    h = hashlib.sha256()
    for f in files:
        with open(os.path.join(PKG, f), "rb") as fh:
            h.update(fh.read())
    assert h.hexdigest()[:16] == m.group(2), f"{name} was taken on other sources than {files}"


def test_every_profile_names_its_command():
    for name in _profiles():
        text = open(os.path.join(PROFILES, name)).read()
        assert "rocprofv3 " in text and "bench.py" in text, name
