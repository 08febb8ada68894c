/*
 * raas_probe.h -- a streaming probe of libraas_probe.so (measurement only;
 * not part of the decode path or of libraas.so).
 *
 * raas_probe_stream reads a buffer laid out as the step kernel's K/V pool
 * (per unit, `tokens` rows of K and of V in 32-token blocks of
 * 32 * head_dim bf16 values each) with the step kernel's access structure
 * and no arithmetic: one workgroup of `waves` wavefronts per unit, each
 * wavefront taking block w, then further blocks claimed from a counter in
 * LDS (dynamic = 1) or a fixed interleave (0), the next block's loads issued
 * before the current block is consumed. mode 0 holds that next block in
 * registers, as the step kernel does; mode 1 stages the blocks in LDS with
 * direct global-to-LDS loads, two 16 KB slots per wavefront (head_dim 128,
 * at most 4 wavefronts). `layers` separate pools are read in turn, one per
 * launch, so that their sum can exceed the memory-side cache; alternate = 1
 * reverses a layer's traversal on every other visit, as the decode path
 * does. kv_interleaved = 1 lays each block's K and V out back to back (one
 * contiguous run per block) instead of in two arrays. The probe allocates
 * and frees its own device memory
 * (units * tokens * head_dim * 4 bytes per layer) and times `launches`
 * launches with HIP events on the default stream after two untimed rounds.
 * Outputs: the average microseconds per launch and the bytes one launch
 * reads. Returns 0, -1 for an invalid configuration, -2 for a failed HIP
 * call.
 */
#ifndef RAAS_PROBE_H
#define RAAS_PROBE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    int32_t units, tokens, head_dim; /* tokens: a multiple of 32; head_dim 64 or 128 */
    int32_t layers;                  /* pools read in turn, >= 1 */
    int32_t waves;                   /* 2, 4 or 8 wavefronts per workgroup */
    int32_t nontemporal;             /* 1: non-temporal loads */
    int32_t mode;                    /* 0: next block in registers; 1: two blocks in LDS slots */
    int32_t dynamic;                 /* 1: dynamic claims after the first block; 0: fixed interleave */
    int32_t alternate;               /* 1: a layer's traversal reverses on every other visit */
    int32_t launches;                /* timed launches, >= 1 */
    int32_t kv_interleaved;          /* 1: a block's K and V halves adjacent (one contiguous run
                                        per block) instead of K and V in separate arrays */
} raas_probe_config;

int raas_probe_stream(const raas_probe_config* cfg, double* us_per_launch, double* bytes_per_launch);

#ifdef __cplusplus
}
#endif

#endif /* RAAS_PROBE_H */
