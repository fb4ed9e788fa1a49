// Build-time tuning of the draw kernels (chosen by measurement on MI355X).
#pragma once

//   LDA_LDS_TABLE_MAX_BLOCKS  largest K / W whose rebuilt table goes to LDS
//                             (see lds_table_for);
//   LDA_WAVES_PER_EU          wavefronts per SIMD the register budget targets;
//   LDA_WAVES_PER_BLOCK       wavefronts per workgroup (for the leaf-group
//                             kernel, 1 and 4 were within 2% of 2 at
//                             K = 16 ... 256).
#ifndef LDA_LDS_TABLE_MAX_BLOCKS
#define LDA_LDS_TABLE_MAX_BLOCKS 0
#endif
#ifndef LDA_WAVES_PER_EU
#define LDA_WAVES_PER_EU 3
#endif
#ifndef LDA_WAVES_PER_BLOCK
#define LDA_WAVES_PER_BLOCK 2
#endif
//   LDA_DOC_LANES_TARGET_WAVES wavefronts the document-per-lane driver aims
//                             for by splitting each group's master loop.
#ifndef LDA_DOC_LANES_TARGET_WAVES
#define LDA_DOC_LANES_TARGET_WAVES 16384
#endif
//   LDA_HALF_MAX_BLOCKS       largest K / 64 for which the W = 64 kernel
//                             rebuilds only the chosen half-block (its 2 K/64
//                             LDS rows per wavefront keep 12 wavefronts per CU
//                             up to 26 blocks, 10 at 32 blocks).
#ifndef LDA_HALF_MAX_BLOCKS
#define LDA_HALF_MAX_BLOCKS 32
#endif
//   LDA_EIGHTHS_MAX_BLOCKS    largest number of 256-topic blocks for which the
//                             leaf kernel with 32-topic prefix rows draws
//                             (8 rows of LDS per block and wavefront; 0: never);
//   LDA_EIGHTHS_SPLIT         largest block count drawn with the first of its
//                             two launch shapes;
//   LDA_EIGHTHS_WINDOW{,_LARGE}, LDA_EIGHTHS_WAVES_PER_EU{,_LARGE}
//                             tokens in flight per wavefront (16-byte loads)
//                             and wavefronts per SIMD of the two shapes.
#ifndef LDA_EIGHTHS_MAX_BLOCKS
#define LDA_EIGHTHS_MAX_BLOCKS 8
#endif
//   LDA_GROUP_MAX_K           largest K drawn by the leaf-group kernel (K
//                             divisible by 4, at most 256; 0: never), and its
//                             tokens in flight per wavefront and wavefronts
//                             per SIMD for groups of 8 to 32 lanes: 8 at 4
//                             (93-118 VGPRs, no spills) was 4-11% faster than
//                             8 at 3 at K = 48 ... 112 and within 2% of the
//                             best of 4 or 8 at 3 ... 5 at K = 16 ... 112.
#ifndef LDA_GROUP_MAX_K
#define LDA_GROUP_MAX_K 256
#endif
#ifndef LDA_GROUP_WINDOW
#define LDA_GROUP_WINDOW 8
#endif
#ifndef LDA_GROUP_WAVES_PER_EU
#define LDA_GROUP_WAVES_PER_EU 4
#endif
//   LDA_GROUP64_WINDOW, LDA_GROUP64_WAVES_PER_EU  the same for groups of 64
//                             lanes (K from 132 to 256): 8 at 3 was 0-15%
//                             faster than 4 at 4, 2 at 4, 16 at 2, 2 or 4 at
//                             5 at K = 144 ... 256.
//   LDA_GROUP_LEAF            topics per lane of the leaf-group kernel (4 or
//                             8: groups of K / 4 or K / 8 lanes, rounded up
//                             to a power of two).
#ifndef LDA_GROUP_LEAF
#define LDA_GROUP_LEAF 4
#endif
//   LDA_GROUP_KEEP_MAX_G      largest group (lanes) of 4-topic leaves that
//                             keeps its leaves' partial sums in LDS for the
//                             final scan instead of reloading the chosen leaf
//                             (0: none).  Groups of 8 (K <= 32): 9-16% faster
//                             at 3-4M tokens (6.75 KiB per wavefront: 22
//                             wavefronts per CU instead of 24); groups of 16:
//                             4-12% slower (12.75 KiB: 12 instead of 20).
#ifndef LDA_GROUP_KEEP_MAX_G
#define LDA_GROUP_KEEP_MAX_G 8
#endif
#ifndef LDA_GROUP64_WINDOW
#define LDA_GROUP64_WINDOW 8
#endif
#ifndef LDA_GROUP64_WAVES_PER_EU
#define LDA_GROUP64_WAVES_PER_EU 3
#endif
//   LDA_LEAF8_MAX_K, LDA_LEAF8_ALIGNED_MAX_K
//                             K above 256 drawn by groups of 64 lanes with
//                             8-topic leaves, the whole row in one tile (K
//                             divisible by 4): up to LDA_LEAF8_MAX_K (at most
//                             512; 0: none), except multiples of 32 above
//                             LDA_LEAF8_ALIGNED_MAX_K; the eighths kernel
//                             draws the rest.  Measured on the 16.8M-token
//                             corpus against the eighths kernel: 17-21%
//                             faster at K = 260 ... 320, 7% at 384, 1-4% at
//                             392 ... 508 (416 included); 2-3% slower at 448,
//                             480 and 512 (rows of whole 128-byte lines).
//   LDA_LEAF8_WINDOW, LDA_LEAF8_WAVES_PER_EU  their tokens in flight per
//                             wavefront and wavefronts per SIMD: 4 at 3
//                             (154-160 VGPRs) was 3-6% faster than 8 at 2 at
//                             K = 260 ... 384 and within 0.5% above; 2 at 4
//                             spills.
#ifndef LDA_LEAF8_MAX_K
#define LDA_LEAF8_MAX_K 508
#endif
#ifndef LDA_LEAF8_ALIGNED_MAX_K
#define LDA_LEAF8_ALIGNED_MAX_K 416
#endif
#ifndef LDA_LEAF8_WINDOW
#define LDA_LEAF8_WINDOW 4
#endif
#ifndef LDA_LEAF8_WAVES_PER_EU
#define LDA_LEAF8_WAVES_PER_EU 3
#endif
//   LDA_EIGHTHS_MIN_K         smallest K it takes (K divisible by 4; the first
//                             block is padded with empty topics up to a
//                             multiple of 256).
#ifndef LDA_EIGHTHS_MIN_K
#define LDA_EIGHTHS_MIN_K 132
#endif
#ifndef LDA_EIGHTHS_SPLIT
#define LDA_EIGHTHS_SPLIT 5
#endif
#ifndef LDA_EIGHTHS_WINDOW
#define LDA_EIGHTHS_WINDOW 16
#endif
#ifndef LDA_EIGHTHS_WAVES_PER_EU
#define LDA_EIGHTHS_WAVES_PER_EU 2
#endif
#ifndef LDA_EIGHTHS_WINDOW_LARGE
#define LDA_EIGHTHS_WINDOW_LARGE 4
#endif
#ifndef LDA_EIGHTHS_WAVES_PER_EU_LARGE
#define LDA_EIGHTHS_WAVES_PER_EU_LARGE 4
#endif
//   LDA_ROUTED_FEW_WINDOW, LDA_ROUTED_FEW_THETA  tokens in flight per
//                             wavefront (phi loads) and theta leaves read
//                             ahead from LDS when a routed wavefront's tokens
//                             form a few runs of documents.
#ifndef LDA_ROUTED_FEW_WINDOW
#define LDA_ROUTED_FEW_WINDOW 16
#endif
#ifndef LDA_ROUTED_FEW_THETA
#define LDA_ROUTED_FEW_THETA 4
#endif
