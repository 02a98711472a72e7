"""MI355X (gfx950) paged attention: varlen chunked prefill + decode over a
block-table KV cache, grouped-query heads, online softmax (arxiv 2511.11581).

``paper_2511_11581_amd.pa`` is the thin ctypes binding of the C-ABI library
``libpa.so`` (declared in ``include/pa.h``); ``workloads`` draws seeded
synthetic batches.  Importing the package loads nothing; the binding loads
the HIP library on first use and raises if it is missing.
"""
