"""CPU oracle for the block-diffusion denoising step and the Redline selection.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this package: only the test-suite, the smoke check in
``__graft_entry__.smoke()`` and the ``cpu_baseline`` leg of ``bench.py`` use it.
It is a plain, slow, deliberately unoptimised restatement of what the paper
defines, written without any code in common with the HIP library.

Modules
  model   -- decoder forward over a window of positions, block-causal attention
             against a KV cache, mask-suppressed LM-head softmax statistics.
  decode  -- the threshold commit rule, in-order commit sweep, admission and
             one-step cache write, as a per-sequence state machine.
  redline -- reference-relative violation counts, exact binomial p-values,
             Holm step-down and the fastest-valid deployment rule.
  quant   -- fp8 E4M3 weight quantization with a power-of-two scale per
             output row (the precision axis of a configuration).

Parity pins (see the tests under ``tests/``) tie every function here to
something other than itself: closed forms, brute force, textbook special
cases and the worked examples printed in the paper.
"""
