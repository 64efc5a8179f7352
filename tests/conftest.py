"""Shared pytest configuration.

Tests marked ``gpu`` run the HIP path on a real MI355X; everything else runs
on the CPU (oracle pins, input-generator checks, host-side library logic).
"""

import os
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)


def pytest_configure(config):
    config.addinivalue_line("markers", "gpu: needs an MI355X (gfx950) GPU and the built HIP library")
