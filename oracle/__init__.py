"""CPU oracle for the paged translate-gather-pack of FlowTrain's unified memory pool.

TEST INFRASTRUCTURE ONLY. Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import or run anything in this package;
the product path (the HIP library and its Python binding) never does, and
shares no code with it.

Plain, slow, obviously correct Python + numpy:

- ``oracle.pack``   the plain definition of a packed microbatch: each
  sample's text rows (embedding-table rows of its ids) and image rows
  interleaved at the image placeholders, samples concatenated, with
  cu_seqlens and per-sample position ids (Sec. 3.1 cross-modal pairing,
  Sec. 4.1 interleaved subsequences, Sec. 3.4 packing into fixed-capacity
  microbatches).
- ``oracle.pool``   a pool with GVA regions and per-rank segments (Sec. 3.2),
  a page table from GVA pages to physical frames in HBM or DRAM tiers, page
  allocators, producer write / free, and a consumer pack that resolves every
  visual row through the page table.
- ``oracle.plan``   the per-sample cost l + l^2/K, the per-microbatch cost of
  Eq. 3, the greedy balanced partition, the zig-zag partition, and
  brute-force optimal partitions.
- ``oracle.allocate`` the heterogeneous parallel allocator of Eq. 1-2:
  pruned candidate configurations and the lexmax (G, -F) flow matching,
  solved by enumerating every combination.
- ``oracle.schedule`` the dynamic packing scheduler of Alg. 1: best-fit
  packing by a plain scan of the open microbatches, Eq. 3 costs, buckets by
  exact one-dimensional k-means, and zig-zag dispatch to ranks.

All arithmetic is on Python ints or numpy integer arrays; embeddings are
moved as raw 16-bit words and never pass through floating point.
"""

from . import allocate, pack, plan, pool, schedule  # noqa: F401
