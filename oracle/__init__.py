"""CPU oracle for the RateQuant hot path -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously-correct reference written from the paper
(arXiv 2605.06675, "RateQuant"), in numpy, fp64 wherever the paper does not
fix a precision.  Only the test-suite, the smoke check and the CPU-baseline
leg of the benchmark may import it; the product library never does, and the
two share no code (only the seeded input generators in ``workloads``).

Modules
  fit        distortion model D(b) = alpha * beta^-b, log-linear OLS
  alloc      reverse waterfilling, greedy integer allocation, brute force
  lloydmax   Lloyd-Max scalar quantizer of N(0,1) (the TurboQuant codebook)
  fmt        fp16/bf16 rounding helpers and the packed code format
  quant      KIVI-, QuaRot-, TurboQuant-style and RTN quantize / dequantize
  cache      residual-window rule and packed-cache assembly for one unit
  attention  fp64 decode attention over a dequantized cache
  calib      per-component distortion sweep
  sensitivity  Stage-1 gradient sensitivity, weight cap, fit fallback
"""
