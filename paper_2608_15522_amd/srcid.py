"""Identity of the library sources: a sha256 over the kernel sources, the
internal headers and the public header, which the build compiles into
libsa.so (``sa_build_id``) and the binding compares on load, so that a
library built from other sources is never called."""
from __future__ import annotations

import hashlib
import os

PKG = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(PKG)
CSRC = os.path.join(PKG, "csrc")
HEADER = os.path.join(ROOT, "include", "sa.h")


def source_files():
    """The files libsa.so is built from, in a fixed order (None if the
    sources are not present next to the package)."""
    if not os.path.isdir(CSRC) or not os.path.exists(HEADER):
        return None
    names = sorted(f for f in os.listdir(CSRC) if f.endswith((".hip", ".h")))
    return [os.path.join(CSRC, f) for f in names] + [HEADER]


def source_id(files=None) -> str | None:
    """First 16 hex digits of the sha256 of the sources (name and bytes of
    each file), or None if they are not present."""
    files = source_files() if files is None else files
    if files is None:
        return None
    h = hashlib.sha256()
    for f in files:
        h.update(os.path.basename(f).encode() + b"\0")
        with open(f, "rb") as fh:
            h.update(fh.read())
        h.update(b"\0")
    return h.hexdigest()[:16]
