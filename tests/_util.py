"""Helpers shared by the tests (no arithmetic of the method)."""
from paper_2502_06798_amd.synth import host_view


def stored_np(t):
    """Host numpy view of a tensor's stored elements (same bytes, same element size)."""
    return host_view(t)


def np_or_none(t):
    return host_view(t)
