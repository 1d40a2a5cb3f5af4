"""CPU oracle of the reuse-aware ViT encoder forward.

TEST INFRASTRUCTURE ONLY.  Only the tests, the smoke check and the bench's
CPU-baseline leg may import this package.  It shares no code with the HIP
path and must never be called from the product path.

Modules:
  reusevit   -- the vectorised oracle (gate mode and mask-injection mode)
  dense_vit  -- an independently written plain ViT forward (no reuse)
  bruteforce -- a per-token loop version of the reuse forward for tiny inputs
"""
from .reusevit import encode, unpack_blob, cosine_rows, gate_decision, reuse_rate  # noqa: F401
from .dense_vit import dense_vit  # noqa: F401
from .bruteforce import encode_bruteforce  # noqa: F401
