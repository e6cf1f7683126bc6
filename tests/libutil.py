"""Loading the built library for tests (builds it first only when nothing is built)."""
import os
import re

from paper_2607_23265_amd import wavezip

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = [os.path.join(ROOT, "include", h) for h in ("wavezip.h", "wavezip_probe.h")]


def ensure_built():
    if not os.path.exists(wavezip.LIB_PATH):
        from paper_2607_23265_amd.csrc import build
        build.build()
    return wavezip.lib()


def declared_functions():
    """Names of the functions the headers under include/ declare."""
    text = "".join(open(h).read() for h in HEADERS)
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(wz_[a-z_]+)\s*\(", text)))
