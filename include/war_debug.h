/*
 * war_debug.h -- diagnostic entry points of libwar.so (not part of the verify path).
 */
#ifndef WAR_DEBUG_H
#define WAR_DEBUG_H

#include "war.h"

#ifdef __cplusplus
extern "C" {
#endif

/* One 16x16x32 bf16 matrix-core product C = A @ B with the lane layout the
 * library's kernels assume.
 *   A  device bf16 [16][32], row-major
 *   B  device bf16 [32][16], row-major
 *   C  device fp32 [16][16], row-major (out)
 * Used by tests to confirm that layout on the hardware; stream-ordered. */
war_status war_debug_mfma16(const void* A, const void* B, float* C, void* stream);

/* Device address and size of one of a model's workspace buffers, for tests that
 * inspect intermediate values after a call (the buffers hold the last layer's
 * values).  Names: "h" fp32 residual [rows][d]; "u" bf16 last norm or SwiGLU
 * output; "q" bf16 rotated queries [rows][nq*hd]; "o" bf16 attention output
 * [rows][nq*hd]; "P" fp32 split-K partials; "pm", "pl", "po" attention
 * partials; "rows", "reqs", "items" step metadata; "order" the attention work
 * order and "n_items" its counts ([0] item slots, [1] units in the work
 * order, [3] keys per attention item, which a verify step's setup chooses:
 * the base length or twice it); "tree" the last tree step's node slots and node masks
 * (int32 [2][max_rows]).  The pointer stays valid until the next call on the
 * model. */
war_status war_debug_workspace(war_model* m, const char* name, void** ptr, int64_t* bytes);

/* The sampled-verification decision kernels alone (those war_verify_step_sampled
 * runs after the LM head), on caller-provided rows: logits device fp32
 * [B*(k_max+1)][V]; ntok device int32 [B] (drafts + 1; 0 = no rows); drafts
 * device int32 [B][k_max]; uniforms, temperature, top_k and the outputs as in
 * war_verify_step_sampled.  Synchronises the stream. */
war_status war_debug_sample(const float* logits, int32_t V, int32_t B, int32_t k_max, const int32_t* ntok,
                            const int32_t* drafts, const float* uniforms, float temperature, int32_t top_k,
                            int32_t* accept_lens, int32_t* next_tokens, void* stream);

/* How many times the pool's verify steps read the exact free page count from
 * the device (each such read waits for the stream) because the host's lower
 * bound did not cover the step's worst-case reservation (HOST out). */
war_status war_debug_pool_waits(war_kv_pool* p, int64_t* waits);

/* Per-kernel timing.  war_profile(m, 1) clears the record and starts timing
 * every kernel launch of later verify/prefill calls on this model.  Each
 * launch is bracketed by a pair of HIP events on the launch stream.
 * war_profile(m, 0) stops.
 * war_profile_read synchronises the device and writes one line per kernel,
 * "name calls total_ms\n", into out (HOST, out_len bytes).  It then clears
 * the record.  The event pairs add a few microseconds per launch, so time
 * whole steps without profiling. */
war_status war_profile(war_model* m, int32_t enable);
war_status war_profile_read(war_model* m, char* out, int32_t out_len);

#ifdef __cplusplus
}
#endif
#endif /* WAR_DEBUG_H */
