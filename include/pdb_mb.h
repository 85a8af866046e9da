/*
 * pdb microbenchmarks: the hardware figures the epoch kernels are priced
 * against on one MI355X (gfx950) -- the streaming copy bandwidth of HBM, the
 * latency of one device-scope hand-over between two compute units, and the
 * cost of one grid-wide barrier.  They do not compute any part of the method;
 * they measure the costs that bound it (a level per barrier, a dependent
 * example per hand-over, an epoch's bytes at the copy rate).  C ABI, same
 * conventions as pdb.h: caller-owned device pointers, work on the caller's
 * stream, PDB_OK or a negative pdb_status.
 */
#ifndef PDB_MB_H
#define PDB_MB_H

#include <stddef.h>
#include <stdint.h>

#include "pdb.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Device workspace (bytes) that pdb_mb_hop and pdb_mb_barrier need. */
int pdb_mb_workspace_bytes(size_t *bytes);

/* Copies `bytes` (a multiple of 16, src and dst 16-byte aligned, not
 * overlapping) from src to dst (device) with one 16-byte load and store per
 * lane per step, a grid-stride loop over every compute unit.  Asynchronous:
 * time it with events on `stream`; read + written bytes over that time is
 * the achievable HBM rate of a plain stream. */
int pdb_mb_copy(const void *src, void *dst, size_t bytes, hipStream_t stream);

/* `rounds` round trips of one 64-bit device-scope word between block 0 and
 * block `partner` (1 .. 1023) of a cooperatively launched grid of one wave
 * per block: block 0 writes 2r + 1 once it reads 2r, the partner writes
 * 2r + 2 once it reads 2r + 1.  Writes the mean time per round trip in
 * nanoseconds (block 0's constant clock) and the XCD of each of the two
 * blocks.  ws: pdb_mb_workspace_bytes().  Synchronous.  A wait that exceeds
 * the watchdog (opt->spin_timeout_us) returns PDB_ERR_DEVICE. */
int pdb_mb_hop(int64_t rounds, int32_t partner, void *ws, size_t ws_bytes, double *ns_per_round,
               int32_t *xcd_a, int32_t *xcd_b, const pdb_options *opt, hipStream_t stream);

/* `rounds` grid-wide barriers (the barrier the level-by-level epoch runs
 * between wide levels: agent-scope release, an arrival counter, a generation
 * word) over a cooperatively launched grid of `blocks` blocks of 256
 * threads.  Writes the mean time per barrier in nanoseconds.  ws:
 * pdb_mb_workspace_bytes().  Synchronous; PDB_ERR_DEVICE when a wait exceeds
 * the watchdog, PDB_ERR_HIP when the grid cannot be resident at once. */
int pdb_mb_barrier(int64_t rounds, int32_t blocks, void *ws, size_t ws_bytes,
                   double *ns_per_barrier, const pdb_options *opt, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* PDB_MB_H */
