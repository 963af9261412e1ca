/*
 * skv_ceiling.h -- streaming reference kernels (libskv_ceiling.so), a
 * measurement aid kept apart from the codec's ABI in skv.h.
 *
 * They report what HBM delivers on this GPU for plain access patterns with
 * the codec's mixes of reads and writes (pack reads about two bytes per byte
 * written, unpack the reverse, and unpack's writes land as 256-byte pieces
 * of the paged cache's token slots).  Bandwidth is not part of the paper's
 * method; these kernels only move bytes.
 */
#ifndef SKV_CEILING_H_
#define SKV_CEILING_H_

#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Access patterns.  `bytes` (a multiple of 128 KiB) sizes every pattern; the
 * bytes each one reads and writes are given by skv_ceiling_bytes. */
enum {
  SKV_CEIL_READ = 0,              /* read `bytes` (16-byte loads)                  */
  SKV_CEIL_WRITE = 1,             /* write `bytes` (16-byte non-temporal stores)   */
  SKV_CEIL_WRITE_DEFAULT = 2,     /* write `bytes` (16-byte default-policy stores) */
  SKV_CEIL_COPY = 3,              /* read and write `bytes`                        */
  SKV_CEIL_READ2_WRITE1 = 4,      /* read `bytes`, write bytes/2 (pack's mix)      */
  SKV_CEIL_READ1_WRITE2_8B = 5,   /* read bytes/2 (8-byte loads), write `bytes`,
                                     both contiguous (unpack's mix)               */
  SKV_CEIL_READ1_WRITE2_16B = 6,  /* the same with 16-byte loads                   */
  SKV_CEIL_NHD_SCATTER = 7,       /* unpack's pattern at d = 128 with 8 heads: one
                                     workgroup per 256-token chunk of a head reads
                                     its 128-byte rows contiguously (bytes/2 in
                                     all) and writes each as 256 bytes into the
                                     token's slot of a [token][8][128] binary16
                                     array (`bytes`), 2 KiB apart               */
  SKV_CEIL_READ1_WRITE4 = 8,      /* read bytes/4 (4-byte loads), write `bytes`
                                     (16-byte default-policy stores), both
                                     contiguous (unpack's mix at INT4)           */
  SKV_CEIL_STAGE_DIRECT = 9,      /* the attention score's key stream: each
                                     workgroup reads 256 KiB into shared memory
                                     in 16 KiB stages, a barrier per stage, with
                                     non-temporal direct global-to-LDS loads
                                     (`bytes` rounded down to 256 KiB; writes
                                     nothing)                                   */
  SKV_CEIL_STAGE_REGS = 10,       /* the same stages loaded into registers
                                     (non-temporal) and written to shared memory
                                     by the threads                             */
  SKV_CEIL_STAGE_DIRECT_CACHED = 11, /* as STAGE_DIRECT with the default cache
                                     policy                                      */
  SKV_CEIL_WRITE_CPOL = 12        /* 12 + p, p in 0..7: write `bytes` with 16-byte
                                     buffer stores whose cache-policy modifiers
                                     are sc0 if p & 1, nt if p & 2, sc1 if p & 4 */
};

/* Enqueues one pass of `pattern` on `stream`, each thread keeping `inflight`
 * (4, 8 or 16) loads in flight before it uses them (the write-only patterns
 * ignore it; the stage patterns keep 1, 2 or 3 stages in flight).  src
 * (device, 16-byte aligned) holds at least the bytes the pattern reads, dst
 * (device) at least the bytes it writes; sink (device, 4 KiB) is needed by
 * SKV_CEIL_READ and the stage patterns only, which store into it only for an
 * input they never see.  Returns 0 on success, 1 for a bad argument (nothing
 * enqueued), 2 if the launch failed. */
int skv_ceiling_run(int32_t pattern, int32_t inflight, void* dst, const void* src, uint64_t bytes, void* sink,
                    hipStream_t stream);

/* Bytes read (which = 0) or written (which = 1) by one call of
 * skv_ceiling_run(pattern, ..., bytes, ...); 0 for an unknown pattern. */
uint64_t skv_ceiling_bytes(int32_t pattern, uint64_t bytes, int32_t which);

#ifdef __cplusplus
}
#endif

#endif /* SKV_CEILING_H_ */
