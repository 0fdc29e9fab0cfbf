"""CPU oracle for the SARA rollout-allocation hot path.

TEST INFRASTRUCTURE ONLY.  Nothing in the product path may import, call, link
or execute this package: only the test-suite, the smoke check and the CPU
baseline leg of the benchmark use it.  It shares no code with the HIP path;
the only common dependency is the seeded input module ``workloads``.

Every function is a plain, slow, direct statement of what the paper (or the
stated reading of it) defines, with no blocking or fusion:

* ``predictor``  - Beta posterior, closed-form predictor p_eff (Prop. 1,
                   Eq. peff) and the two-threshold rule (Eq. decide).
* ``controller`` - one allocation step (Algorithm 1) as a slot-pool event
                   simulation on the decode-step clock.
* ``philox``     - Philox4x32-10 counter-based generator (Salmon et al., SC'11).
* ``sampler``    - temperature + Gumbel-max token draw over the top-p
                   nucleus, forced-EOS draw.
* ``reward``     - synthetic verifiable reward: SplitMix64-finalizer hash chain
                   over the generated tokens, thresholded against p_uid.
* ``model``      - pre-norm GQA decoder (RMSNorm, RoPE, SwiGLU) with bf16
                   rounding at the storage points the bf16 configs use.
* ``grpo``       - group-relative advantages (Eq. grpo).
* ``run``        - a full allocation step: controller + lazily generated rollouts.

Parity status of each part is listed in the module headers; the transformer
has no value printed in the paper and is pinned by independent checks.
"""
