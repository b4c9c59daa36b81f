"""Compiled structured-sparse decoder runtime for MI355X (gfx950).

``binding`` exposes the C ABI of ``libtasp.so`` (include/tasp.h) under the same names;
``session`` builds the ABI structs around torch-owned device memory. Importing the package does
not load the library; the first call does, and fails loudly if it has not been built.
"""
from . import binding  # noqa: F401

__all__ = ["binding"]
