"""Plain CPU oracle for the reservoir-fed surrogate training path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call or run
anything in this package; only the tests, the smoke check and the benchmark's
CPU-baseline leg do.  It shares no code with the HIP library: it is written
from the paper (Algorithm 1 "Reservoir" and Sec. 3.2.3 for the buffer, Sec. 4.1
for the surrogate and its Adam training) and from the published definition of
the Philox counter-based generator.

Modules:
  philox     -- Philox4x64-10 and the integer range map used for every draw.
  reservoir  -- slot encoding of Algorithm 1 (put with eviction of seen items,
                batch draw with replacement, threshold, drain after reception).
  buffers    -- the FIFO and FIRO comparison buffers of Sec. 3.2.3 (samples
                leave the buffer when read).
  mlp        -- fp64 MLP forward, mean-squared-error loss, backward, Adam, with
                an optional bf16 operand-rounding mode.
  runner     -- the deterministic put / sample / train loop over a workload.

Parity status per function is listed in each module header.
"""
