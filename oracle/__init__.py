"""CPU oracle for the SSM block-wise denoising step.

TEST INFRASTRUCTURE ONLY.  Only the test suite, the smoke check and the
benchmark's CPU-baseline leg may import this package; the product path never
does and has no CPU fallback.  It shares no code with the HIP path.

Plain, slow NumPy (float64 unless a caller asks for float32 to fit the 8B
shapes in host memory).  Every function cites the passage of the paper it
follows.  Where the paper is silent the reading taken is stated in the
function's docstring.

Modules
  selection  suffix partition and retention, compacted row list  (Sec. 3.2, Eq. 1-5)
  embed      top-k renormalisation, soft embedding, mixing       (Sec. 3.2, Eq. 6-8)
  model      bidirectional transformer step with prefix KV cache (Sec. 3.2 sparse input)
  unmask     confidence-based unmasking rules                    (Sec. 4.2)
  generate   block-wise generation loop                          (Sec. 3.2, Sec. 4)
"""
from . import selection, embed, model, unmask, generate  # noqa: F401
