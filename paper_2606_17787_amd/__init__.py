"""MI355X-native paged KV-cache checkpoint and restore (LUMEN's data path).

Modules:
  kvckpt     Python binding of the HIP library (include/lumen_kv_ckpt.h)
  build      in-tree hipcc build of the library for gfx950
  workloads  seeded synthetic inputs (cache shapes, ranges, block tables)

Importing the package loads nothing; the library is loaded on first use.
"""
