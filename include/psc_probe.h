/* psc_probe.h -- libpsc_probe.so: a measurement aid beside the mask library,
 * not part of the mask path.  It times the kind of load the classifier walk
 * (Algorithm 2, the classification step) makes: a chain of dependent loads
 * through a table, in the fused step's launch shape.
 */
#ifndef PSC_PROBE_H
#define PSC_PROBE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    PSC_PROBE_WAVE_LOAD = 0,    /* 16 bytes per lane, 1 KiB per wavefront: a sparse row's or chain's load */
    PSC_PROBE_SCALAR_LOAD = 1   /* one 8-byte load at a uniform address: a dense row's entry (scalar path) */
};

/* Enqueue one launch on `stream` (a hipStream_t) and return a hipError_t
 * (0 on success; hipErrorInvalidValue for an argument out of range, before any
 * launch: an unknown mode, n_rows < 1, k < 0, grid_y over 65,535, more than
 * 2^24 workgroups, or fill without out).  Grid grid_x x grid_y workgroups of
 * four wavefronts; wavefront 0 of each makes k dependent loads through
 * `table`, device memory of n_rows rows
 * of 256 int32 (1 KiB) each, caller-owned: the first row is a hash of the
 * workgroup and `seed`, each next row the magnitude of a loaded value modulo
 * n_rows.  Then, when fill != 0, the four wavefronts store 4 KiB each to
 * `out` (device memory of grid_x * grid_y * 16 KiB, caller-owned;
 * nontemporal device-scope stores, as the step's logits stores).  A launch
 * with k = 0 times everything but the chain, so (t(k) - t(0)) / k is the
 * latency of one dependent load.  Asynchronous; nothing is allocated. */
int psc_probe_chase(int32_t mode, void *out, const int32_t *table, int32_t n_rows, int32_t k, int32_t fill,
                    int32_t grid_x, int32_t grid_y, uint32_t seed, void *stream);

#ifdef __cplusplus
}
#endif

#endif
