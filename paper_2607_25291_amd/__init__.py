"""CoSA prefill attention for MI355X (gfx950): KAP proxy + ordered-skipping kernel, C-ABI library.

The HIP library is loaded lazily by ``paper_2607_25291_amd.binding``; importing the package itself
touches neither the GPU nor the library.
"""
