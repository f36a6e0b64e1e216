"""Shared helpers for tests that touch the built library."""
import os
import re

from paper_2607_21604_amd import akvs

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "akvs.h")


def ensure_built():
    """Load libakvs.so; build it first only if nothing is built."""
    if not os.path.exists(akvs.LIB_PATH):
        from paper_2607_21604_amd import build
        build.build()
    return akvs.load()


def declared_functions():
    """Names of the functions include/akvs.h declares (return type, name, parameter list)."""
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(akvs_[a-z_0-9]+)\s*\(", text)))
