"""Locate (and on a CPU-only machine, build) libhxf.so for the tests."""
import os

from paper_2505_05286_amd import hxf


def ensure_built():
    if os.path.exists(hxf.LIB_PATH):
        return hxf.LIB_PATH
    from paper_2505_05286_amd import build
    return build.build()
