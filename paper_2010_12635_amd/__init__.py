"""GCN layer forward/backward on MI355X (gfx950): hand-written HIP kernels
behind the C-ABI library ``libgcn.so``.  ``paper_2010_12635_amd.gcn`` is the
Python binding (argument marshalling only)."""
