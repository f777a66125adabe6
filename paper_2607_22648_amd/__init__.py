"""MI355X-native hot path of PTStore's prefix store.

``libptstore.so`` (HIP, gfx950) holds the whole path: chained block hashing,
the open-addressing block index with parent links, the batched longest
common prefix lookup, KV gather / scatter between the store's pool and a
paged cache, and the deduplicating insert. ``ptstore`` is its Python binding
(import it explicitly; importing this package loads nothing).
"""
