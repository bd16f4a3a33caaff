"""MI355X-native ARC-KV per-context KV-cache compaction (gfx950 HIP kernels behind a C ABI)."""
from . import arckv  # noqa: F401
