"""Oracle: plain, slow, obviously-correct CPU definitions (TEST INFRASTRUCTURE).

Only tests/, __graft_entry__.smoke() and bench.py's cpu_baseline leg may
import anything from this package.  The HIP path (paper_2607_11136_amd) never
imports it and shares no code with it.

Modules
  block   fp64 numpy definition of one DiT block forward (Secs. 2.1, 2.2, 5.2)
  brute   the same definition as scalar pure-Python loops, for tiny shapes
  layout  Algorithm 1 (Sec. 6.1) and the "only as much as needed" chunk plan
          (Sec. 5.1, the pi* objective) over the block's slot table
  offload the selective weight-offloading plan of an N-block step (Sec. 5.1)
  step    an N-block step: the blocks applied in sequence (Sec. 2.1)
  vae     the VAE decoder's upsampling stage (Secs. 2.1, 5.2): nearest 2x
          upsampling, then a 3x3 convolution (reading R25)

Readings.  The paper names the DiT block but prints none of its arithmetic, so
the following conventions are readings (they bind the oracle and the HIP path
alike):
  R1  one shared weight set for text and visual tokens (single-stream block);
      R24 is the dual-stream variant
  R2  m = W_ada c + b_ada (no SiLU), split (shift1, scale1, gate1, shift2,
      scale2, gate2); modulation xhat (1 + scale) + shift; residual x + gate * y
  R3  LayerNorm without affine, biased variance, eps 1e-6
  R4  QK-RMSNorm per head over d, gains shared by all heads, eps 1e-6, applied
      before RoPE
  R5  RoPE theta 10000, head vector split in contiguous [t | y | w] segments
      of widths (d_t, d_h, d_w), interleaved pairs (2j, 2j+1), integer
      positions from 0; text tokens and dims past the segments unrotated
  R6  token order: text first, then visual tokens t-major, then y, then w
  R7  full bidirectional joint attention, no mask, scale 1/sqrt(d)
  R8  GELU in its tanh form
  R9  every Linear has a bias
  R10 conditioning width D_c = D
  R11 synthetic inputs (see the workloads package)
  R17 Algorithm 1 tie-breaks (see layout)
  R25 VAE upsampling stage: nearest-neighbour 2x, then 3x3 convolution with
      zero padding 1 and bias, NHWC activations, weight [C_out, 3, 3, C_in]
  R24 dual-stream modulation: a block may carry a second AdaLN map
      (ada_txt_w, ada_txt_b) whose split modulates the text tokens (positions
      below L_t); the visual tokens keep m; every other weight is shared
  R28 the block's slot table follows the implementation's intermediates: at
      head_dim 64 the QKV projection writes Q, K and V^T directly, so the
      [tokens, 3D] qkv slot is empty (layout.block_tensors)

Parity pins: see tests/test_oracle_pins.py and tests/test_layout_oracle.py.
The conventions R2, R5, R6, R9-R11 are fixed by no value the paper prints, so
the oracle is pinned to them only through its own invariants and the
independent scalar version ("parity unpinned" for those conventions).
"""
