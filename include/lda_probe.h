/*
 * lda_probe.h -- C ABI of the measurement probes (liblda_probe.so), gfx950.
 *
 * These kernels draw nothing.  They move memory the way the draw does, or
 * the way a plain stream does, so that the draw's time can be set against
 * what the memory system allows:
 *
 *   lda_probe_draw_floor  a memory-only copy of the draw's access pattern
 *                         (the leaf kernels of lda_draw_butterfly, for K
 *                         divisible by 4 up to 2048): every token's phi row
 *                         read once as 16-byte leaves (64 lanes read 1 KiB of
 *                         one row per load), the theta row of each run of one
 *                         document's tokens read once, u read and z written,
 *                         in the same token order and wavefront grid, with no
 *                         arithmetic beyond summing what it loads.  Its time
 *                         is the floor of a draw that moves the method's
 *                         compulsory bytes in token order (the draw itself
 *                         also rereads the chosen part of each row).
 *   lda_probe_read        a streaming read of a buffer, `passes` times over:
 *                         with a buffer larger than the 256 MiB MALL the
 *                         bytes come from HBM; with one larger than the L2s
 *                         (8 x 4 MiB) but inside the MALL, the passes after
 *                         the first are served by the MALL: the rate at which
 *                         L2 misses can be served at all.
 *
 * Statuses, pointer ownership and streams as in lda_draw.h (device pointers
 * owned by the caller; calls only enqueue on `stream`).  The probes write
 * only their output (z, or out).
 */
#ifndef LDA_PROBE_H
#define LDA_PROBE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * Memory-only floor of the draw.  Arguments as lda_draw_butterfly (theta
 * [M][K], phi [V][K], doc_id, word_id, u [N], z [N] written with a value of
 * no meaning), plus:
 *   window          16-byte loads issued per wavefront before their values
 *                   are summed: 8 or 16;
 *   waves_per_group wavefronts per workgroup: 2 or 4;
 *   waves_per_cu    0: as many wavefronts per CU as fit; 1 ... 32: at most
 *                   that many (an LDS allocation per workgroup caps them), to
 *                   match a draw whose registers allow no more.
 * Rows of K <= 256 topics are read by groups of G = 8, 16, 32 or 64 lanes
 * (G the smallest with 4 G >= K, as the draw), so one load reads the rows of
 * 64 / G tokens; longer rows in blocks of 256 topics, one token per load.
 * Leading leaves that fall before topic 0 (K not a multiple of the row
 * width) load topic 0's leaf, as the draw does.
 * K must be divisible by 4 with 4 <= K <= 2048 and N >= 64, else
 * LDA_ERR_UNSUPPORTED; other errors as lda_draw_butterfly.
 */
int lda_probe_draw_floor(const float *theta, const float *phi, const int32_t *doc_id,
                         const int32_t *word_id, const float *u, int32_t *z, int64_t N,
                         int32_t M, int32_t V, int32_t K, int32_t window,
                         int32_t waves_per_group, int32_t waves_per_cu, void *stream);

/*
 * Streaming read: `passes` times over, every 16 bytes of buf[0 .. bytes)
 * are read once and summed (LDA_PROBE_READ_GROUPS workgroups of 256 lanes,
 * all resident at once, each reading a contiguous span with 16 loads of 16
 * bytes in flight per lane); each lane writes its sum to out
 * (float [LDA_PROBE_READ_OUT_FLOATS]).  buf 16-byte aligned and bytes a
 * multiple of 16 (LDA_ERR_ALIGN), passes >= 1 and bytes >= 0
 * (LDA_ERR_SHAPE); bytes = 0 is a no-op.
 */
#define LDA_PROBE_READ_GROUPS 2048
#define LDA_PROBE_READ_OUT_FLOATS (LDA_PROBE_READ_GROUPS * 256)
int lda_probe_read(const void *buf, int64_t bytes, int32_t passes, float *out, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* LDA_PROBE_H */
