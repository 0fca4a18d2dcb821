"""MI355X-native cached mixed-precision EmbeddingBag training step.

The compute path lives in HIP kernels behind the C ABI declared in
``include/emb_cache.h`` (library ``paper_2010_11305_amd/libembcache.so``);
``paper_2010_11305_amd.emb_cache`` is the thin ctypes binding.  Importing this
package loads nothing; the binding loads the library on first use and raises if
it has not been built.
"""
__all__ = ["configs", "workload", "emb_cache"]
