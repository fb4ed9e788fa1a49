/*
 * lda_draw.h -- C ABI of the MI355X (gfx950) per-token LDA topic draw.
 *
 * Method: G. L. Steele Jr. and J.-B. Tristan, "Using Butterfly-Patterned
 * Partial Sums to Optimize GPU Memory Accesses for Drawing from Discrete
 * Distributions" (arXiv 1505.03851).
 *
 * The operation (Section 2, problem statement and Algorithm 1): for every
 * token n with document d = doc_id[n] and word w = word_id[n], topic k has the
 * relative weight a_k = theta[d][k] * phi[w][k].  With S_k = a_0 + ... + a_k
 * and S = S_{K-1}, the draw is
 *
 *     z[n] = the smallest k with u[n] * S < S_k            (strict "<")
 *
 * and K - 1 when no k qualifies (S = 0, or u*S rounding up to S), which is
 * what the linear and binary searches of Algorithms 2 and 3 return.  The
 * arithmetic is fp32; a result may differ from exact arithmetic only for
 * tokens whose u*S lies within fp32 rounding of some S_k.
 *
 * Layout (all arrays dense and row-major, as Section 3 assumes):
 *   theta   float [M][K]  document-topic weights, a document's K topics
 *                         contiguous; entries >= 0 and finite.
 *   phi     float [V][K]  topic-word weights stored word-major: row w holds
 *                         word w's weight in every topic, K contiguous floats
 *                         (the paper's phi[V, K]); entries >= 0 and finite.
 *   doc_id  int32 [N]     0 <= doc_id[n] < M; need not be sorted (tokens of one
 *                         document stored contiguously run faster).
 *   word_id int32 [N]     0 <= word_id[n] < V.
 *   u       float [N]     the uniform variate of each draw, 0 <= u[n] < 1.  The
 *                         paper draws it inside the procedure; here the caller
 *                         supplies it.
 *   z       int32 [N]     output topics, 0 <= z[n] < K.
 *
 * Ownership and memory: every pointer is a device pointer (hipMalloc'd, or
 * memory that the caller's framework allocated on the current device),
 * owned by the caller, 4-byte aligned.  The library keeps no state between
 * calls and allocates no device memory; kernels use on-chip LDS only (and,
 * in the naive kernel, the per-lane private segment the HIP runtime manages).
 * The routed draw keeps its routing, and the indexed counts their word
 * index, in a workspace the caller provides (lda_draw_routed_scratch: in a
 * static array the library holds).
 *
 * Streams: `stream` is a hipStream_t (NULL = the default stream).  Calls only
 * enqueue work and return; the caller synchronises (lda_route_build alone
 * waits, once, for its first kernels, to read back the word class counts).
 * Calls that share the output buffer must be ordered by the caller.
 *
 * Errors: every entry point returns LDA_OK (0) or a negative status.  Argument
 * checks happen before any HIP call, so a rejected call has no effect and
 * touches no device.  N == 0 is a no-op returning LDA_OK (the counts: tables
 * cleared).  Preconditions that are not checked (ids in range, finite
 * non-negative weights, u in [0, 1)) are the caller's: an out-of-range id
 * gives a meaningless draw, and in lda_draw_naive and lda_butterfly_table,
 * which address theta and phi directly, reads outside them (the other draws
 * read through range-checked buffer resources, or past 4 GiB clamp the id to
 * the last row).
 */
#ifndef LDA_DRAW_H
#define LDA_DRAW_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LDA_OK 0
#define LDA_ERR_NULL (-1)        /* a required pointer is NULL while N > 0   */
#define LDA_ERR_SHAPE (-2)       /* N < 0, M <= 0, V <= 0 or K <= 0          */
#define LDA_ERR_UNSUPPORTED (-3) /* K > LDA_MAX_K, N > LDA_MAX_N, or a table
                                    too large                                */
#define LDA_ERR_HIP (-4)         /* the HIP runtime reported an error        */
#define LDA_ERR_ALIGN (-5)       /* a pointer is not 4-byte aligned          */
#define LDA_ERR_WORKSPACE (-6)   /* routing workspace too small or mismatched */

/* Largest number of topics the kernels accept. */
#define LDA_MAX_K 4096

/* Largest number of tokens: a launch holds about one work-item per token, and
 * a dispatch counts its work-items in 32 bits (2^32 - 2^16).  Token indices
 * are 64-bit throughout.  Larger N is rejected with LDA_ERR_UNSUPPORTED. */
#define LDA_MAX_N 4294901760LL

/* Largest size in bytes of theta (4*M*K) or phi (4*V*K) for most entry
 * points: their kernels address both through buffer
 * resources, whose record count and byte offsets are unsigned 32-bit.  Larger
 * tables are rejected with LDA_ERR_UNSUPPORTED. */
#define LDA_MAX_TABLE_BYTES 4294967295LL

/* lda_draw_butterfly, lda_draw_docs and lda_draw_butterfly_philox take theta
 * and phi of any size (M and V below 2^31): when either table is larger than
 * LDA_MAX_TABLE_BYTES they draw with a second build of the same kernels that
 * addresses rows by index and forms 64-bit addresses (ids beyond the table's
 * rows are clamped to its last row there, so no read leaves the table); the
 * draws are the same.
 *
 * Largest size in bytes of both count tables of lda_count_topics, and of
 * nwk in lda_count_topics_docs and lda_count_topics_indexed: 2^32 - 1 cells
 * (16 GiB; those cells are keyed by unsigned 32-bit indices).  The latter two
 * take ndk of any size (M below 2^31): its rows are written whole at 64-bit
 * addresses. */
#define LDA_MAX_COUNT_TABLE_BYTES 17179869180LL

/*
 * Baseline draw: Algorithm 1 with the binary search of Algorithm 3.  One lane
 * per token; each lane walks its own theta and phi rows (lanes of a wavefront
 * read addresses 4*K bytes apart), keeps the full prefix table of its token in
 * its private segment and binary-searches it.
 */
int lda_draw_naive(const float *theta, const float *phi, const int32_t *doc_id,
                   const int32_t *word_id, const float *u, int32_t *z,
                   int64_t N, int32_t M, int32_t V, int32_t K, void *stream);

/*
 * Butterfly draw (Algorithm 7 with Algorithms 5, 8, 9 and 10, Sections 3-4).
 * A wavefront takes 64 consecutive tokens, one per lane, and reads theta and
 * phi cooperatively: each load instruction fetches consecutive topics of one
 * token, or of a few tokens (coalesced), instead of one topic of 64 tokens.
 * The lanes combine their products in a butterfly pattern (log2 W exchange
 * stages) instead of a full transposition, and each lane reconstructs the
 * partial sums it needs from the butterfly table while it searches for u*S
 * (Algorithm 10).  The kernel depends on K:
 *  - K divisible by 4 up to 256 (N >= 64): groups of W = 8, 16, 32 or 64
 *    lanes, each lane one leaf of 4 topics; load k brings token k's whole
 *    row into its group; the butterfly runs over the W leaf sums, Algorithm
 *    10 finds the token's leaf and a scan of its 4 products the topic
 *    (groups of 8 lanes keep each leaf's partial sums in LDS for that scan;
 *    the others read the leaf again); from 260 to 508 (multiples of 32 only
 *    up to 416) the same with 64 lanes and leaves of 8 topics;
 *  - K divisible by 4 from 260 to 2048 otherwise: 256-topic blocks read as leaves of 4
 *    topics per lane; a first sweep keeps every token's prefix at the end of
 *    each 32-topic part of each block, Algorithm 9 finds the part holding
 *    u*S, whose butterfly table is rebuilt on chip and searched;
 *  - otherwise: blocks of W topics, one topic per lane (W = 64 for K >= 64,
 *    32 below), the prefix at each block end, then Algorithm 9 and the
 *    rebuilt block (or half-block) with Algorithm 10.
 * Where K is not a multiple of the block (or of the group's 4 W topics), the
 * first K mod block topics (the remnant) form a leading block padded with
 * empty topics, which are never drawn.  theta and phi may be of any size
 * (past LDA_MAX_TABLE_BYTES the same kernels run with 64-bit table
 * addressing).
 */
int lda_draw_butterfly(const float *theta, const float *phi,
                       const int32_t *doc_id, const int32_t *word_id,
                       const float *u, int32_t *z, int64_t N, int32_t M,
                       int32_t V, int32_t K, void *stream);

/*
 * Butterfly draw over documents given in the paper's ragged form (Section 2:
 * document m holds N[m] tokens; Algorithm 7 draws document by document):
 * doc_offsets is an int64 device array [M + 1], non-decreasing, with
 * doc_offsets[0] = 0 and doc_offsets[M] = N; document m's tokens are
 * word_id[doc_offsets[m] .. doc_offsets[m+1]), with their u and z at the same
 * positions.  Empty documents are allowed.  The result equals
 * lda_draw_butterfly with doc_id[n] = the document whose range holds n.
 * Tokens are still drawn one per lane, 64 consecutive tokens per wavefront:
 * each lane finds its document by binary search over doc_offsets.
 * doc_offsets must be 8-byte aligned (LDA_ERR_ALIGN otherwise); its contents
 * are not checked.  Tables of any size, as lda_draw_butterfly.
 */
int lda_draw_docs(const float *theta, const float *phi,
                  const int64_t *doc_offsets, const int32_t *word_id,
                  const float *u, int32_t *z, int64_t N, int32_t M, int32_t V,
                  int32_t K, void *stream);

/*
 * The paper's document-per-lane driver (Algorithm 7): 64 consecutive
 * documents form a group, one per lane, and a master index walks their
 * tokens in step; a lane whose document has run out repeats its last token
 * (without storing) until the group's longest document is done.  Each
 * group's master loop is split over several wavefronts (index i = s, s + S,
 * ...) so that the launch fills the GPU.  Arguments, layout and errors as
 * lda_draw_docs (doc_offsets int64 [M + 1], 8-byte aligned; out-of-range
 * offsets are clamped to [0, N], never dereferenced), plus:
 *   theta_cache  0: theta is read from memory in every iteration;
 *                1: Algorithm 5's cache -- each wavefront first copies its
 *                   documents' theta rows into LDS in transposed order; only
 *                   for K up to LDA_DOC_LANES_MAX_CACHE_BYTES / 256 rounded
 *                   to whole blocks (K <= 256), else LDA_ERR_UNSUPPORTED.
 * Same z as lda_draw_docs except inside the fp32 rounding band (the lanes
 * sum in another order).  Slower than lda_draw_docs: it is provided to
 * measure the paper's design.
 */
#define LDA_DOC_LANES_MAX_CACHE_BYTES 65536
int lda_draw_doc_lanes(const float *theta, const float *phi,
                       const int64_t *doc_offsets, const int32_t *word_id,
                       const float *u, int32_t *z, int64_t N, int32_t M, int32_t V,
                       int32_t K, int32_t theta_cache, void *stream);

/*
 * Butterfly draw with the uniforms generated in the kernel (Algorithm 1's
 * draw of u inside the procedure; the paper names no generator): token n
 * takes u = (y >> 8) * 2^-24, y the first output word of Philox4x32-10
 * (Salmon, Moraes, Dror and Shaw, SC 2011) with key (seed mod 2^32,
 * seed >> 32) and counter (n mod 2^32, n >> 32, sweep, 0).  Arguments,
 * layout, dispatch and errors as lda_draw_butterfly without u; a caller
 * passes a new `sweep` (or seed) for every pass over the corpus.  The
 * result equals lda_draw_butterfly given u from lda_philox_uniforms.
 */
int lda_draw_butterfly_philox(const float *theta, const float *phi,
                              const int32_t *doc_id, const int32_t *word_id,
                              int32_t *z, int64_t N, int32_t M, int32_t V,
                              int32_t K, uint64_t seed, uint32_t sweep, void *stream);

/*
 * The uniforms lda_draw_butterfly_philox uses, written out: u[i] (device,
 * float32 [count], 4-byte aligned) = uniform of token first + i for `seed`
 * and `sweep`.  count = 0 is a no-op; negative count or first, or
 * first + count past INT64_MAX, is LDA_ERR_SHAPE.
 */
int lda_philox_uniforms(float *u, int64_t count, int64_t first, uint64_t seed,
                        uint32_t sweep, void *stream);

/*
 * Butterfly draw with a chosen per-block table, for measuring the table's
 * design choices (Section 4).  Same arguments, layout and errors as
 * lda_draw_butterfly, plus `variant`:
 *   LDA_VARIANT_REGISTER_TABLE  the paper's replacement [a b; c d] ->
 *                               [a d; a+b c+d]; the table stays in registers
 *                               and Algorithm 10's search-assist loop fetches
 *                               each level's entry with cross-lane reads;
 *   LDA_VARIANT_LDS_TABLE       the same table written to LDS; each search
 *                               level reads its entry directly;
 *   LDA_VARIANT_LDS_TABLE_ALT   the alternative rule the paper mentions,
 *                               [a b; c d] -> [a c; a+b c+d], whose table
 *                               holds left-half sums of aligned topic ranges,
 *                               searched in LDS by a descent from the whole
 *                               block;
 *   LDA_VARIANT_LEAF8           where lda_draw_butterfly uses its leaf groups
 *                               (K divisible by 4 up to 256, N >= 64), leaves
 *                               of 8 topics per lane in groups half as wide;
 *                               elsewhere the kernels of lda_draw_butterfly;
 *   LDA_VARIANT_WIDE_TABLES     the kernels of lda_draw_butterfly as built for
 *                               tables past 4 GiB (rows by index, 64-bit
 *                               loads), at any table size: the same draws as
 *                               lda_draw_butterfly, to compare the two builds.
 * The three table variants use the one-topic-per-lane kernel for all K
 * (W = 64 for K >= 64, else 32).  Any other `variant` returns
 * LDA_ERR_UNSUPPORTED.
 */
#define LDA_VARIANT_REGISTER_TABLE 0
#define LDA_VARIANT_LDS_TABLE 1
#define LDA_VARIANT_LDS_TABLE_ALT 2
#define LDA_VARIANT_LEAF8 3
#define LDA_VARIANT_WIDE_TABLES 4
int lda_draw_butterfly_variant(const float *theta, const float *phi,
                               const int32_t *doc_id, const int32_t *word_id,
                               const float *u, int32_t *z, int64_t N, int32_t M,
                               int32_t V, int32_t K, int32_t variant, void *stream);

/*
 * Transposed-access draw (Algorithms 4, 5 and 6 with a binary search over
 * block ends and a linear search of the chosen block, Section 3): the
 * paper's design before the butterfly, kept for comparison.  The tile of W =
 * 64 topics x 64 tokens is read with the same coalesced loads as
 * lda_draw_butterfly, then transposed through LDS so that each lane sums its
 * own token's products in topic order (16.6 KiB of LDS per wavefront).  Same
 * arguments, layout, errors and result as lda_draw_butterfly.
 */
int lda_draw_transposed(const float *theta, const float *phi,
                        const int32_t *doc_id, const int32_t *word_id,
                        const float *u, int32_t *z, int64_t N, int32_t M,
                        int32_t V, int32_t K, void *stream);

/*
 * The butterfly-patterned tables themselves (Section 4, Fig. 1 right), for
 * inspection and tests.  table is a device float array [N][K]: row n is the
 * table p[K] that token n's lane holds in Algorithm 7 -- the remnant's full
 * prefix, then for each block of W topics the W-1 butterfly entries of that
 * lane's column followed by the full prefix at the block's end.  Entries of a
 * column sum products of the other tokens of the same group of W lanes (lane
 * groups are tokens [g*W, g*W + W), the last group padded by repeating token
 * N-1).  W is chosen from K as in lda_draw_butterfly.
 */
int lda_butterfly_table(const float *theta, const float *phi,
                        const int32_t *doc_id, const int32_t *word_id,
                        float *table, int64_t N, int32_t M, int32_t V,
                        int32_t K, void *stream);

/*
 * Tokens routed to the GPU's XCDs by word.  The MI355X dispatches workgroups
 * to its eight XCDs round robin, and each XCD has its own L2.  In token order
 * every XCD reads phi rows from the whole vocabulary; routing gives every XCD
 * the tokens of one eighth of the vocabulary, so its L2 serves more of them.
 * The draw is the same per token (Algorithms 7-10 with 16-byte leaf loads);
 * only the grouping of tokens into wavefronts changes.  Routing pays where
 * phi is far larger than the caches and costs where phi fits the 256 MiB
 * MALL.  Measured on MI355X over 16.8M Zipf tokens with V = 100,000 words:
 * 28% slower than lda_draw_butterfly at K = 256, 3% slower at K = 512, 4%
 * faster at K = 768, 6% at K = 1024, 13% at K = 2048 (28% on 9.8M tokens
 * with V = 50,000 at K = 2048); so lda_draw_routed takes K >= LDA_ROUTE_MIN_K
 * only.
 *
 * lda_route_build: splits the words into 256 classes by a hash, assigns the
 * classes to 8 lists with about equal token counts, and lays the tokens out
 * in the caller's workspace as those 8 lists, each in the original token
 * order and padded to a multiple of 64.  It depends on doc_id and word_id
 * only, so a sampler builds it once per corpus and reuses it every sweep.
 * It enqueues the class count on `stream` and synchronises `stream` once to
 * read the counts back (the one entry point that waits; it cannot be
 * captured into a HIP graph, while lda_draw_routed can); the host then
 * assigns the classes, fills *route and enqueues the layout's kernels, which
 * a draw on the same stream follows (a draw on another stream needs the
 * caller's synchronisation).
 *   workspace        device memory, 8-byte aligned, at least
 *                    lda_route_workspace_bytes(N) bytes (about 12.25 N), owned
 *                    by the caller; it holds the routing and must stay
 *                    unchanged until the last lda_draw_routed that uses it.
 *   route            host struct filled on success.
 * Errors as above; LDA_ERR_WORKSPACE if workspace_bytes is too small;
 * LDA_ERR_UNSUPPORTED if N > LDA_ROUTE_MAX_N.
 *
 * lda_draw_routed: the draw of lda_draw_butterfly over routed tokens: z[n]
 * and u[n] are indexed by the original token n.  theta, phi, M, V, K as for
 * lda_draw_butterfly; K must be divisible by 4 with LDA_ROUTE_MIN_K <= K <=
 * 2048, else LDA_ERR_UNSUPPORTED (below, use lda_draw_butterfly); `route` and `workspace` must come from one
 * lda_route_build over these N tokens, else LDA_ERR_WORKSPACE.
 *
 * lda_draw_routed_philox: lda_draw_routed with the uniforms generated in the
 * kernel exactly as lda_draw_butterfly_philox does (Philox4x32-10 of the
 * original token index, sweep and seed), so its z equals that entry point's
 * z except inside the rounding band.
 */
#define LDA_ROUTE_MAX_N 2147483135LL
#define LDA_ROUTE_MIN_K 768
typedef struct lda_route {
  int64_t N;          /* tokens routed */
  int64_t tokens[8];  /* tokens in list x */
  int64_t start[8];   /* first routed position of list x */
  int64_t length[8];  /* positions of list x: tokens[x] rounded up to 64 */
} lda_route;

size_t lda_route_workspace_bytes(int64_t N);
int lda_route_build(const int32_t *doc_id, const int32_t *word_id, int64_t N, int32_t M,
                    int32_t V, void *workspace, size_t workspace_bytes, lda_route *route,
                    void *stream);
int lda_draw_routed(const float *theta, const float *phi, const void *workspace,
                    size_t workspace_bytes, const lda_route *route, const float *u,
                    int32_t *z, int64_t N, int32_t M, int32_t V, int32_t K, void *stream);
int lda_draw_routed_philox(const float *theta, const float *phi, const void *workspace,
                           size_t workspace_bytes, const lda_route *route, int32_t *z,
                           int64_t N, int32_t M, int32_t V, int32_t K, uint64_t seed,
                           uint32_t sweep, void *stream);

/*
 * Topic counts of a set of draws: the statistics the update of theta and
 * phi consumes once every z has been drawn (Section 1: a topic is drawn for
 * every word from theta and phi, then theta and phi are updated; Section 2:
 * the uncollapsed sampler whose draw phase the other entry points perform).
 *   ndk[d][k] = number of tokens n with doc_id[n] = d and z[n] = k
 *   nwk[w][k] = number of tokens n with word_id[n] = w and z[n] = k
 * ndk is int32 [M][K] and nwk int32 [V][K] (word-major, the layout of phi),
 * row-major device arrays owned by the caller; both are overwritten (zeroed
 * first, also when N = 0).  doc_id, word_id and z are int32 [N] device
 * arrays (z typically the output of a draw on the same stream).  A token
 * whose document, word or topic lies outside [0, M), [0, V) or [0, K) is not
 * counted.  Integer work: the result is exact and does not depend on the
 * order of the tokens.  Every pointer 4-byte aligned (LDA_ERR_ALIGN); ndk and
 * nwk may not be NULL (LDA_ERR_NULL), nor the token arrays when N > 0;
 * N above LDA_COUNT_MAX_N (counts are int32), K above LDA_MAX_K, or either
 * table above LDA_MAX_COUNT_TABLE_BYTES (2^32 - 1 cells: cells are addressed
 * by unsigned 32-bit indices) give LDA_ERR_UNSUPPORTED.  Enqueues two
 * kernels that clear the tables, then one that counts; nothing is allocated.
 */
#define LDA_COUNT_MAX_N 2147483647LL
int lda_count_topics(const int32_t *doc_id, const int32_t *word_id, const int32_t *z,
                     int64_t N, int32_t M, int32_t V, int32_t K, int32_t *ndk, int32_t *nwk,
                     void *stream);

/*
 * lda_count_topics with the documents in the paper's ragged form (Section 2:
 * document m holds N[m] tokens), as lda_draw_docs takes them: doc_offsets is
 * an int64 device array [M + 1], non-decreasing, doc_offsets[0] = 0 and
 * doc_offsets[M] = N, 8-byte aligned (LDA_ERR_ALIGN); document m's tokens are
 * positions doc_offsets[m] .. doc_offsets[m+1] - 1 of word_id and z.  The
 * result equals lda_count_topics with doc_id[n] = the document whose range
 * holds n.  The documents being contiguous, each row of ndk is counted by
 * one wavefront and written whole: ndk needs no clearing and no atomics in
 * memory (K <= LDA_MAX_K bins of LDS per wavefront).  Offsets outside [0, N]
 * are clamped, never dereferenced; their contents are not otherwise checked.
 * Other arguments and errors as lda_count_topics, except that ndk may be of
 * any size (only nwk above LDA_MAX_COUNT_TABLE_BYTES gives
 * LDA_ERR_UNSUPPORTED); doc_offsets may not be NULL (also when N = 0).
 */
int lda_count_topics_docs(const int64_t *doc_offsets, const int32_t *word_id, const int32_t *z,
                          int64_t N, int32_t M, int32_t V, int32_t K, int32_t *ndk,
                          int32_t *nwk, void *stream);

/*
 * A word index of the tokens, for the topic counts of many sweeps over one
 * corpus (the word ids do not change between sweeps; the counts do): the
 * positions of each word's tokens, built once by a counting sort on the GPU.
 * The caller provides `index`, device memory of at least
 * lda_word_index_bytes(N, V) bytes, 8-byte aligned (LDA_ERR_ALIGN), which
 * the index occupies until the caller frees it; the library keeps no state.
 * Layout inside it, each section on a 256-byte boundary: off int32 [V + 1]
 * (the positions of word w are off[w] .. off[w+1] - 1; off[V] = the tokens
 * indexed), the build's per-word counters int32 [16 V] (one to a 64-byte
 * line), the scan's workgroup sums, perm
 * int32 [N] (the token at each position) and wsorted int32 [N] (its word).
 * Tokens whose word id lies outside [0, V) are not indexed.  The order of a
 * word's tokens is not fixed; the counts do not depend on it.
 * lda_word_index_bytes returns 0 for N < 0, V <= 0, N > LDA_COUNT_MAX_N or
 * V > LDA_WORD_INDEX_MAX_V.  The build enqueues seven kernels on `stream`
 * (no memset, no wait: it may be captured into a graph); word_id int32 [N]
 * device, 4-byte aligned, NULL only when N = 0; errors LDA_ERR_SHAPE (N < 0,
 * V <= 0), LDA_ERR_UNSUPPORTED (N > LDA_COUNT_MAX_N, V >
 * LDA_WORD_INDEX_MAX_V), LDA_ERR_NULL, LDA_ERR_ALIGN, LDA_ERR_WORKSPACE
 * (index_bytes too small).
 */
#define LDA_WORD_INDEX_MAX_V 16777215
size_t lda_word_index_bytes(int64_t N, int32_t V);
int lda_word_index_build(const int32_t *word_id, int64_t N, int32_t V, void *index,
                         size_t index_bytes, void *stream);

/*
 * lda_count_topics_docs with the word table counted from a word index
 * (lda_word_index_build over the same word_id, N and V): the tokens are taken
 * word by word, each workgroup a run of 2,048-position chunks; each cell's
 * tokens are summed in an LDS table, and when the table is written out the
 * cells of a word whose tokens all lie in the positions summed since the last
 * write are stored, the others (words that straddle writes or workgroups)
 * added with device atomics.  Same results as lda_count_topics_docs
 * (exact); same arguments and errors, plus those of the index
 * (LDA_ERR_WORKSPACE when index_bytes < lda_word_index_bytes(N, V)).  An index
 * built from other tokens gives wrong counts but no access outside ndk, nwk,
 * the index and the token arrays.
 */
int lda_count_topics_indexed(const int64_t *doc_offsets, const int32_t *word_id,
                             const int32_t *z, int64_t N, int32_t M, int32_t V, int32_t K,
                             const void *index, size_t index_bytes, int32_t *ndk, int32_t *nwk,
                             void *stream);

/*
 * For callers that cannot allocate device memory (code under graph capture
 * aside: this call waits on the stream; tight serving loops; harnesses that
 * forbid hipMalloc): lda_route_build followed by lda_draw_routed, with the
 * routing kept in a scratch array the library holds instead of a caller's
 * workspace.  Arguments, layout, errors and z as lda_draw_routed (K divisible
 * by 4 with LDA_ROUTE_MIN_K <= K <= 2048), taking doc_id and word_id in
 * place of a route.  The array is a static device array of
 * LDA_ROUTED_SCRATCH_BYTES: each GPU the library runs on holds its own copy
 * until the process ends; N whose routing needs more
 * (lda_route_workspace_bytes(N) > LDA_ROUTED_SCRATCH_BYTES, about 5.4M
 * tokens) is refused with LDA_ERR_UNSUPPORTED before any HIP call.  Nothing
 * is allocated (no hipMalloc, no hipFree).  Like lda_route_build it
 * synchronises `stream` once.  Every call on one GPU uses that GPU's array
 * and overwrites the previous call's routing; calls that overlap on one GPU
 * (other streams, other host threads) race and must be ordered by the
 * caller.
 */
#define LDA_ROUTED_SCRATCH_BYTES 67108864
int lda_draw_routed_scratch(const float *theta, const float *phi, const int32_t *doc_id,
                            const int32_t *word_id, const float *u, int32_t *z, int64_t N,
                            int32_t M, int32_t V, int32_t K, void *stream);

/* The W (butterfly width) the library uses for K, or LDA_ERR_UNSUPPORTED /
 * LDA_ERR_SHAPE for a K it rejects. */
int lda_butterfly_width(int32_t K);

/* A static, human-readable description of a status code. */
const char *lda_status_string(int status);

/* The HIP error string behind the last LDA_ERR_HIP returned on this host
 * thread ("no error" if none). */
const char *lda_last_hip_error(void);

/* Library version, as major * 10000 + minor * 100 + patch. */
int lda_version(void);

#ifdef __cplusplus
}
#endif

#endif /* LDA_DRAW_H */
