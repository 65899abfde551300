"""Oracle for the speculative-verification decode step -- TEST INFRASTRUCTURE ONLY.

A plain, slow, obviously-correct CPU implementation (numpy, float64) of what the
HIP path computes.  Only ``tests/``, ``__graft_entry__.smoke()`` and the
``cpu_baseline`` leg of ``bench.py`` may import it; the product path never
does, and this package imports nothing from the product package.

Modules
  bf16      round-to-nearest-even to bfloat16, written from the IEEE-754 format.
  decoder   the GQA decoder forward over a block of new tokens against a
            request's cached keys/values (dense, per request, row by row).
  accept    greedy argmax (ties -> lowest id) and longest-matching-prefix
            acceptance of draft tokens.
  pages     the paged-KV bookkeeping model: free stack, refcounts, block tables,
            reserve / commit / rollback / fork / free.
  verify    one verify step / one prefill-append for a batch, composed from the
            above in the order the method takes them.
  sampling  sampled verification (temperature, top-k, lossless speculative
            sampling with a deterministic drafter; uniforms are inputs).

What the paper fixes (arXiv 2607.17299):
  * speculative decoding is lossless: the target model verifies drafts and the
    output matches what the target alone would produce (Introduction; Background,
    "Why Workload Matters");
  * drafts proposed by the suffix-tree drafter are verified by the target model in
    one forward pass, advancing several tokens when accepted (System Design,
    "SuffixDecoding"); with speculation off the step is plain batched decode
    (System Design, "SuffixDecoding", adaptive enabling and stateless mode switching);
  * new turns are appended to a trajectory whose KV cache is reused (System Design,
    "Overview of WAR"; Background, "Rollout Bottlenecks").
The paper names no acceptance rule, decoder, KV layout or precision; the readings
taken for those points are greedy exact-match acceptance and the decoder below
(RMSNorm, rotate-half RoPE, grouped-query attention, SwiGLU, untied LM head).
"""
