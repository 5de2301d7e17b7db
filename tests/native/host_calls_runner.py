"""Run pytest with the library's host-only calls taken from a separately
built copy of their sources (argv[1], e.g. a sanitizer build) instead of
libtempokv.so; argv[2:] are pytest arguments.  Used by tests/test_sanitizers.py
in a child process."""
import ctypes as ct
import os
import sys

ROOT = os.path.dirname(os.path.dirname(os.path.dirname(os.path.abspath(__file__))))
sys.path.insert(0, ROOT)

import paper_2609_35065_amd as kv  # noqa: E402

kv._host_override = kv.declare(ct.CDLL(sys.argv[1]), kv.HOST_CALLS)

import pytest  # noqa: E402

rc = pytest.main(["-x", "-q", "-p", "no:cacheprovider", *sys.argv[2:]])
if rc == 0 and kv._lib is not None:
    print("libtempokv.so was loaded: a selected test did not go through the host calls' copy")
    rc = 3
sys.exit(rc)
