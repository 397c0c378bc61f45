"""MI355X-native DeDLOC averaging round: shard reduce, wire codecs and LAMB.

The compute runs in the HIP library `libdedloc.so` (built from `csrc/`);
`paper_2106_10207_amd.dedloc` is the thin ctypes binding over its C ABI.
Importing this package loads nothing; the binding loads the library on first
use and raises if it is missing."""
