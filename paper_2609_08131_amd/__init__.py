"""MI355X (gfx950) implementation of the Jacap eviction scoring path.

``paper_2609_08131_amd.jacap`` binds the C ABI of ``libjacap.so`` (built by
``paper_2609_08131_amd.build``); it is not imported here so that the package can
be imported to build the library.
"""

__all__ = ["jacap", "build"]
