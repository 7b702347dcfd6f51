/*
 * dora_measure.h — measurement entry points of libdora.
 *
 * They are not part of the method.  They let a benchmark time the kernels of
 * one decode call separately, and compare the decode kernel with a plain
 * streaming read that has the decode kernel's access pattern (random 4 KiB
 * tiles, 16-byte non-temporal loads): the achievable-bandwidth reference next
 * to the HBM peak in the decode kernel's roofline.  The conventions of dora.h
 * hold here too (caller-owned device memory, errors before any launch,
 * asynchronous on `stream`).
 */
#ifndef DORA_MEASURE_H
#define DORA_MEASURE_H

#include "dora.h"

#ifdef __cplusplus
extern "C" {
#endif

/* dora_decode_attn with per-kernel timing.  Same arguments, results and
 * errors as dora_decode_attn, plus `events`: three caller-created hipEvent_t
 * (non-NULL) recorded on `stream` before the first decode kernel (events[0]),
 * between it and its combine kernel (events[1]) and after the last combine
 * kernel (events[2]).  DORA_ERR_INVALID_ARG if events or one of its entries is
 * NULL.  No event is recorded when an error is returned before any launch. */
dora_status dora_decode_attn_timed(const dora_decode_desc* desc,
                                   const void* q, const void* k_pages, const void* v_pages,
                                   const int32_t* block_table, const int32_t* seq_lens,
                                   const int32_t* version_ids, void* out,
                                   void* workspace, size_t workspace_bytes,
                                   dora_stream_t stream, void* const* events);

/* Streaming-read reference kernel.  Reads n_tiles tiles of tile_bytes bytes,
 * tile i starting at base + tiles[i] * tile_bytes, with 16-byte non-temporal
 * loads.  `waves` one-wavefront workgroups each take an equal contiguous range
 * of the tile list (the first n_tiles mod waves ranges one tile more), read it
 * in batches of tiles_per_batch tiles with two batches in flight, and fold
 * every word they read into one 32-bit XOR, written to sink[w] (so that no
 * load is dead).
 *   base        device, 16-byte aligned, base_bytes bytes
 *   tiles       device int32 [n_tiles]; a tile that does not lie inside
 *               [base, base + base_bytes) contributes nothing (its loads go to
 *               the buffer's first 16 bytes)
 *   tile_bytes  1024, 2048, 4096, 8192 or 16384
 *   tiles_per_batch  1, 2, 4, 8 or 16, with tile_bytes * tiles_per_batch at
 *               most 16384 (else, like another tile_bytes, DORA_ERR_UNSUPPORTED)
 *   sink        device uint32 [waves]
 *   waves       >= 1
 * n_tiles = 0 writes 0 to every sink word. */
dora_status dora_stream_read(const void* base, int64_t base_bytes, const int32_t* tiles,
                             int64_t n_tiles, int32_t tile_bytes, int32_t tiles_per_batch,
                             uint32_t* sink, int32_t waves, dora_stream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* DORA_MEASURE_H */
