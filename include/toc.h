/*
 * toc.h -- C ABI of libtoc: tuple-oriented compression (TOC) of mini-batches and
 * matrix products run directly on the compressed form, on one MI355X (gfx950).
 *
 * Method: Li et al., "Tuple-oriented Compression for Large-scale Mini-batch
 * Stochastic Gradient Descent" (arXiv 1702.06943).
 *
 * Conventions shared by every call
 *  - Columns are 0-based.  Values, W, G, R and out are IEEE binary32.
 *  - Every call returns a toc_status; on anything but TOC_OK, toc_last_error()
 *    gives a message (thread-local).  No call aborts, exits or throws.
 *  - Handles (toc_enc, toc_dev) are allocated and freed by the library and are
 *    immutable once created: concurrent calls on one handle from several host
 *    threads are allowed, as are device calls on distinct streams.
 *  - Device memory (the upload buffer, W, G, R, out, workspaces, decoded CSR) is
 *    always allocated and owned by the caller.  `stream` is a hipStream_t passed
 *    as void* (NULL = the null stream).  Device calls only enqueue work: they are
 *    asynchronous with respect to the host, and every argument is checked on the
 *    host before anything is enqueued.
 */
#ifndef TOC_H
#define TOC_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  TOC_OK = 0,
  TOC_EINVAL = 1,       /* invalid argument: shape, pointer, CSR form, value      */
  TOC_ENOMEM = 2,       /* host allocation failed                                 */
  TOC_ESIZE = 3,        /* caller's buffer (upload buffer, workspace) too small   */
  TOC_EDEVICE = 4,      /* HIP runtime reported an error (copy, launch)           */
  TOC_EUNSUPPORTED = 5  /* valid, but beyond a documented limit of this build     */
} toc_status;

/* Host-side encoded mini-batch: the pair (I, D) of Algorithm 1. */
typedef struct toc_enc toc_enc;
/* Host descriptor of batches uploaded into a caller-owned device buffer. */
typedef struct toc_dev toc_dev;

typedef struct {
  int32_t n_rows;       /* rows of the mini-batch                                 */
  int32_t n_cols;       /* columns (m)                                            */
  int64_t nnz;          /* column_index:value pairs kept (zeros dropped)          */
  int64_t n_first;      /* |I|: distinct pairs = first layer of the prefix tree   */
  int64_t n_codes;      /* |D|: codes over all rows                               */
  int64_t n_nodes;      /* |C'| including the root = 1 + |I| + sum(len(D_i)-1)    */
  int64_t n_live;       /* codes referenced by D plus their ancestors             */
  int64_t n_deep;       /* live codes whose sequence has two or more pairs        */
  int32_t max_depth;    /* longest live sequence                                  */
  int32_t reserved;
  int64_t phys_bytes;   /* size of the paper's physical encoding (section 3.2)   */
  int64_t canon_bytes;  /* canonical compressed bytes:
                           4|D| + 4(n_rows+1) + 10 n_live + 4(max_depth+1)       */
} toc_enc_info;

/* ---------------------------------------------------------------------------
 * Encoding (host).  Section 3: sparse encoding, then the logical encoding of
 * Algorithm 1 (PrefixTreeEncode): phase I makes every distinct pair a child of
 * the root in order of first appearance, phase II encodes each tuple by greedy
 * longest matches in the prefix tree and grows the tree by one node after every
 * match that does not end the tuple.
 *
 * Input is one mini-batch as CSR: rowptr[n_rows+1] (rowptr[0] == 0, non-
 * decreasing), col[rowptr[n_rows]] strictly increasing inside each row and in
 * [0, n_cols), val[rowptr[n_rows]] finite.  Entries equal to zero (+0.0 or -0.0)
 * are dropped, as the sparse encoding ignores zeros.  Pairs compare equal when
 * column and the binary32 bit pattern of the value are equal.
 * Errors: TOC_EINVAL for any violation above or NULL pointers (col/val may be
 * NULL when rowptr[n_rows] == 0); TOC_EUNSUPPORTED when a batch would need more
 * than 2^31-1 tree nodes; TOC_ENOMEM.  *out is NULL unless TOC_OK.
 * The input arrays are read only during the call.
 * ------------------------------------------------------------------------- */
toc_status toc_encode(int32_t n_rows, int32_t n_cols, const int64_t *rowptr,
                      const int32_t *col, const float *val, toc_enc **out);

/* Encode n_batches mini-batches held in one concatenated CSR, in parallel on
 * n_threads host threads (<= 0: all hardware threads).  Batch b owns the
 * n_rows[b] rows that follow those of batches 0..b-1; rowptr has
 * sum(n_rows)+1 entries and rowptr[0] == 0.  Each batch is encoded on its own
 * exactly as toc_encode would (its own prefix tree; section 3.1).  out[] receives
 * n_batches handles; on any error none is kept and all out[b] are NULL. */
toc_status toc_encode_batches(int64_t n_batches, const int32_t *n_rows, int32_t n_cols,
                              const int64_t *rowptr, const int32_t *col,
                              const float *val, int32_t n_threads, toc_enc **out);

/* Sizes and counts of an encoded batch (see toc_enc_info). */
toc_status toc_enc_info_get(const toc_enc *enc, toc_enc_info *info);

/* Copy out (I, D) in the numbering of Algorithm 1 (node 0 is the root, I holds
 * nodes 1..|I|).  I_col/I_val: n_first entries; D_rowptr: n_rows+1 entries
 * (offsets into D_codes); D_codes: n_codes entries.  Any pointer may be NULL to
 * skip that array.  Host memory, caller-owned. */
toc_status toc_enc_export(const toc_enc *enc, int32_t *I_col, float *I_val,
                          int64_t *D_rowptr, uint32_t *D_codes);

void toc_enc_free(toc_enc *enc);

/* ---------------------------------------------------------------------------
 * Upload.  Rebuilds the decoding tree C' of each batch from (I, D) with
 * Algorithm 2 (section 4.1.2), derives each node's depth, keeps the live codes
 * (those referenced by D and their ancestors; the others take part in no
 * operation of section 4), orders them by depth so that every parent precedes its
 * children, renumbers parents and D, and writes the result into `buf` as one
 * structure-of-arrays image laid out as described by toc_layout below.
 *
 * All batches must have the same n_cols.  toc_upload_size gives the bytes `buf`
 * needs; toc_upload builds the image range of batches by range of batches into
 * two pinned host staging buffers of 256 MiB (or of the largest batch, if
 * larger) in turn, copying each range with hipMemcpyAsync on `stream` while the
 * next is built, and waits for the copies, so the handles in `encs` may be freed
 * afterwards and host memory never holds the whole image.  `buf` must stay
 * allocated for as long as the returned toc_dev is used.
 * flags: TOC_UPLOAD_KEEP_DEAD keeps every node of C' (results are identical);
 *        TOC_UPLOAD_HOST writes the image into host memory `buf` without any HIP
 *        call (for inspection; device operations reject such a toc_dev).
 * Errors: TOC_EINVAL (NULL, n_batches < 0, mismatched n_cols, unknown flag),
 * TOC_ESIZE (bytes < toc_upload_size), TOC_EUNSUPPORTED (a batch above 2^31-1
 * codes or rows), TOC_EDEVICE, TOC_ENOMEM.
 * ------------------------------------------------------------------------- */
#define TOC_UPLOAD_KEEP_DEAD 1u
#define TOC_UPLOAD_HOST 2u

toc_status toc_upload_size(const toc_enc *const *encs, int64_t n_batches,
                           uint32_t flags, size_t *bytes);
toc_status toc_upload(const toc_enc *const *encs, int64_t n_batches, uint32_t flags,
                      void *buf, size_t bytes, void *stream, toc_dev **out);
void toc_dev_free(toc_dev *dev); /* frees the descriptor only, never `buf` */

typedef struct {
  int64_t n_batches;
  int64_t n_rows;        /* sum of rows over batches (rows of R, G, CSR)           */
  int32_t n_cols;        /* m                                                      */
  int32_t max_depth;     /* over all batches                                       */
  int64_t nnz;           /* pairs over all batches (decoded CSR size)              */
  int64_t n_codes;       /* |D| over all batches                                   */
  int64_t n_stored;      /* codes stored in the image (live, or all with KEEP_DEAD)*/
  int64_t n_deep;        /* stored codes of depth >= 2                             */
  int64_t canon_bytes;   /* sum of toc_enc_info.canon_bytes                        */
  int64_t image_bytes;   /* bytes of the uploaded image                            */
} toc_dev_info;

toc_status toc_dev_info_get(const toc_dev *dev, toc_dev_info *info);

/* Byte offsets (from `buf`) of the arrays of the uploaded image.  Codes of batch b
 * are local indices 0..n_codes-1, stored from code_base; local code c is at
 * depth d when level[lvl_base+d-1] <= c < level[lvl_base+d] (level[lvl_base] = 0).
 * Depth-1 codes come first; among them the n_int1 codes that have children
 * precede the others.  The left multiplication reads codes at positions: a
 * depth-1 code without children (a leaf) is at position n_int1 + its rank in
 * (key column, code) order, every other code at its own index.
 *   batches : toc_batch[n_batches]
 *   level   : uint32 per batch n_levels+1 entries (lvl_base)
 *   key     : toc_key of each code (its key pair, 8 bytes), so that a code's key
 *             comes with one 8-byte read
 *   link    : toc_link of each code of depth >= 2 (its parent and depth, 8 bytes),
 *             code c of batch b at deep_base + c - n_lvl1; a depth-1 code has none
 *             (no parent, depth 1)
 *   span    : uint32 per batch n_rows+1 offsets into the batch's D (span_base)
 *   dcodes  : uint32 local code of each entry of D (d_base)
 *   occ_off : uint32 per batch n_codes+2 entries (at code_base + 2 b): first,
 *             for each leaf position p = n_int1 .. n_lvl1 (the last one the end),
 *             where position p's leaf occurrences start in the batch's centry;
 *             then, for each tree row h = 0 .. n_tree (h as in tchild, the last
 *             the end), where tree code h's occurrences start.  A code's
 *             occurrences are the tuples holding it: D inverted, the index set of
 *             the sum that defines G(x) in Theorem 2
 *   tlist   : uint32 per batch the codes with children or of depth >= 2, sorted
 *             by key column (tree_base)
 *   dtiles  : uint32 x 4 per run of 1024 entries of D (at least one per batch):
 *             batch, first entry, pairs of the batch before that entry, first
 *             row whose span starts at or after that entry
 *   cols    : uint32 per batch 4 (n_cols+1) entries (at b * 4 (n_cols+1)): for each
 *             column j = 0..n_cols, the first position of a leaf whose key column
 *             is >= j, the leaf occurrences (centry entries) of such leaves
 *             before it, and the first tlist entry of key column >= j; then the columns
 *             ordered by number of such occurrences plus tree codes, most first
 *             (n_cols entries and one unused)
 *   tchild  : uint32 per batch n_tree+1 entries (at tree_base + b): the children of
 *             tree code h (h counting the codes with children at depth 1, then
 *             the codes of depth >= 2) are the codes tchild[h] .. tchild[h+1]-1
 *   centry  : uint32 per batch n_d + n_tree entries (at d_base + tree_base), in
 *             three parts: (1) the leaf occurrences, leaf by leaf in position
 *             order (so a column's leaves are one stretch, from its cols entry),
 *             each leaf's tuples ascending with bit 31 set on its first; (2) the
 *             tree codes (tlist entries) by key column, each with bit 30 set,
 *             column j's from (1)'s end plus its cols tlist entry; (3) the tree
 *             codes' own occurrences, tree row by tree row (plain tuple indexes,
 *             ascending), where occ_off points.  Needs rows and codes below 2^30
 *             per batch.
 *   cval    : float per centry entry (same index): in parts (1) and (2) the key
 *             value of the entry's code (the multiplier of the left
 *             multiplication's term), 0 in part (3)
 * Depth-1 codes without children are numbered in the order of their first entry
 * in D; the codes of each level d >= 2 are sorted by parent.                    */
typedef struct {
  int64_t code_base, d_base, row_base, span_base, nnz_base, deep_base, tree_base,
      lvl_base;
  int32_t n_rows, n_codes, n_lvl1, n_int1, n_levels, n_d;
  int32_t n_ucols;   /* distinct key columns of the batch's stored codes           */
  int32_t pad;
} toc_batch;

/* A node of the decoding tree C' (Algorithm 2): its key pair (section 3.1) ... */
typedef struct {
  uint32_t col;      /* key column                                               */
  float val;         /* key value                                                */
} toc_key;

/* ... and its place in the tree. */
typedef struct {
  uint32_t parent;   /* local code of the parent; 0xFFFFFFFF at depth 1           */
  uint32_t depth;    /* length of the node's sequence                            */
} toc_link;

typedef struct {
  int64_t batches, level, key, link, span, dcodes, occ_off, tlist, dtiles, cols, tchild, centry,
      cval, end;
} toc_layout;

toc_status toc_dev_layout_get(const toc_dev *dev, toc_layout *layout);

/* ---------------------------------------------------------------------------
 * Device operations.  Workspace: toc_workspace_size gives the bytes an op needs
 * to run in one pass over all batches; an op given less (but at least its
 * per-batch minimum, returned in *min_bytes when not NULL) runs in several
 * passes; less than the minimum is TOC_ESIZE.  A size of 0 means ws may be NULL.
 * The workspace is scratch: its contents on entry do not matter.
 * op: TOC_OP_RIGHT, TOC_OP_LEFT, TOC_OP_DECODE.
 * ------------------------------------------------------------------------- */
#define TOC_OP_RIGHT 0
#define TOC_OP_LEFT 1
#define TOC_OP_DECODE 2

toc_status toc_workspace_size(const toc_dev *dev, int32_t op, int32_t k,
                              size_t *bytes, size_t *min_bytes);

/* Right multiplication R = A.W on every batch (Theorem 1; Algorithm 4 for k = 1,
 * Algorithm 7 for a matrix): the dictionary table H[c] = H[parent(c)] +
 * val(c) W[col(c), :] built level by level over C', then R[i, :] = sum of H over
 * the codes of tuple i.  W: n_cols x k, row-major with row stride ldw >= k.
 * R: (sum of rows) x k, row stride ldr >= k, rows stacked in batch order.
 * Errors: TOC_EINVAL (k < 1, strides, NULL, host-image toc_dev), TOC_ESIZE,
 * TOC_EDEVICE. */
toc_status toc_right_mul(const toc_dev *dev, const float *W, int32_t k, int64_t ldw,
                         float *R, int64_t ldr, void *ws, size_t ws_bytes,
                         void *stream);

/* Left multiplication G^T.A on every batch (Theorem 2; Algorithm 5 for k = 1,
 * Algorithm 8 for a matrix): scatter G rows onto the codes of each tuple,
 * propagate child to parent in reverse depth order, and accumulate
 * val(c) H[c, :] into out[col(c), :].  The result is stored transposed, one
 * n_cols x k block per batch: out[(b n_cols + j) ldo + q] = (G_b^T A_b)[q, j].
 * G: (sum of rows) x k, row stride ldg >= k.  accumulate != 0 adds into out
 * instead of overwriting it.  Errors as toc_right_mul. */
toc_status toc_left_mul(const toc_dev *dev, const float *G, int32_t k, int64_t ldg,
                        float *out, int64_t ldo, int32_t accumulate, void *ws,
                        size_t ws_bytes, void *stream);

/* Left multiplication without any allocation, for callers that cannot allocate
 * device memory (work captured into a HIP graph, tight serving loops, harnesses
 * that forbid hipMalloc).  The same product as toc_left_mul, bit for bit, with no
 * workspace argument: the workspace is a static device buffer of
 * TOC_NOALLOC_SCRATCH_BYTES that the library holds on every GPU it runs on until
 * the process ends (its address is looked up on the first call on each device).
 * When the full grid's per-worker slots do not fit in it, fewer persistent
 * workers run (slower, same result).  Calls on one GPU share that buffer: calls
 * that overlap in time on one GPU (other streams, other host threads) race and
 * must be ordered by the caller.  Nothing in the buffer needs to be zero on entry.
 * Allocates nothing (no hipMalloc, hipFree, or allocating library call).
 * Errors: as toc_left_mul; TOC_EUNSUPPORTED when one batch's workspace (one worker
 * slot per XCD, or one batch's rows on the fallback path) exceeds the buffer. */
#define TOC_NOALLOC_SCRATCH_BYTES (64u << 20)
toc_status toc_left_mul_noalloc(const toc_dev *dev, const float *G, int32_t k, int64_t ldg,
                                float *out, int64_t ldo, int32_t accumulate, void *stream);

/* Full decode of every batch to one CSR (the backtracking of Algorithm 6, without
 * its densify step): rowptr[(sum of rows)+1] (int64), col[nnz] (int32),
 * val[nnz] (float, bit-identical to the encoded values).  Rows in batch order.
 * Errors: TOC_EINVAL, TOC_EDEVICE. */
toc_status toc_decode_csr(const toc_dev *dev, int64_t *rowptr, int32_t *col,
                          float *val, void *stream);

/* Sparse-safe element-wise operation on every batch, in place (section 4.2,
 * Algorithm 3: every distinct key pair of A is a node key of the image, so
 * changing the key values changes every nonzero of A alike).  Each key value v
 * becomes v * c (TOC_MAP_SCALE) or v * v (TOC_MAP_SQUARE; c is ignored), rounded
 * to binary32; the products and decodes that follow see the new matrix.  A value
 * that becomes 0 stays a stored entry.  The image bytes in the caller's buffer are
 * modified; the toc_dev descriptor is not.  Asynchronous on `stream`.
 * Errors: TOC_EINVAL (unknown op, non-finite c, NULL or host-image toc_dev),
 * TOC_EDEVICE. */
#define TOC_MAP_SCALE 0
#define TOC_MAP_SQUARE 1
toc_status toc_map_values(const toc_dev *dev, int32_t op, float c, void *stream);

/* Sparse-unsafe element-wise plus (section 4.5, Algorithm 9): every batch decoded
 * to dense and c added to every element, the zeros included:
 * A[i lda + j] = a_ij + c (binary32) for i < sum of rows (rows in batch order) and
 * j < n_cols; columns n_cols .. lda-1 are left untouched.  A: caller-owned device
 * memory of (sum of rows) x lda floats, lda >= n_cols.  With c = 0 this is the
 * densify step of the algorithm alone.  Asynchronous on `stream`.
 * Errors: TOC_EINVAL (NULL, lda < n_cols, non-finite c, host-image toc_dev),
 * TOC_EDEVICE. */
toc_status toc_decode_dense(const toc_dev *dev, float c, float *A, int64_t lda, void *stream);

/* ---------------------------------------------------------------------------
 * Physical encoding and the decoding tree on the device.
 *
 * Section 3.2 stores (I, D) as bytes: bit packing (ceil(log2(max+1)/8) bytes per
 * integer, behind a header with the count and the bytes per integer) and value
 * indexing of I's values.  The paper leaves the byte layout open; this library
 * reads it as five arrays, in order: I's columns, the unique values (the distinct
 * binary32 bit patterns of I's values, ascending, 4 bytes each), I's value
 * indexes, D's codes of all tuples concatenated (paper numbering), the tuple
 * starts (n_rows + 1 offsets into D, the last one |D|).  Each array is a 5-byte
 * header (count: little-endian u32; bytes per integer: u8, 1..4, 4 for the
 * values) followed by count little-endian integers of that many bytes.
 * ------------------------------------------------------------------------- */
typedef struct {
  int64_t n_rows;       /* tuples                                                 */
  int64_t n_first;      /* |I|                                                    */
  int64_t n_codes;      /* |D|                                                    */
  int64_t n_unique;     /* distinct values of I                                   */
  int64_t n_nodes;      /* |C'| including the root = 1 + |I| + sum(len(D_i)-1)    */
  int64_t max_col;      /* largest column of I (-1 when I is empty): the blob is for
                           a matrix of more than max_col columns                  */
} toc_phys_info;

/* Bytes of the physical encoding of one encoded batch (host, synchronous). */
toc_status toc_enc_pack_size(const toc_enc *enc, size_t *bytes);
/* Writes them to dst (host memory of at least that many bytes): TOC_ESIZE if
 * bytes is smaller. */
toc_status toc_enc_pack(const toc_enc *enc, void *dst, size_t bytes);
/* Reads the headers, I's columns and the tuple starts of one blob in host memory
 * and checks the layout (sizes, widths, starts non-decreasing from 0 to |D|):
 * TOC_EINVAL if it does not hold.  max_col lets the caller check the blob against
 * its matrix's columns before any device step.  Codes and value indexes are
 * checked by toc_cprime_build. */
toc_status toc_phys_info_get(const void *blob, size_t bytes, toc_phys_info *info);

/* Workspace bytes of toc_cprime_build for n_batches batches and n_nodes nodes in
 * total. */
toc_status toc_cprime_workspace_size(int64_t n_batches, int64_t n_nodes, size_t *bytes);

/* Algorithm 2 (BuildPrefixTree, section 4.1.2) on the device, one workgroup per
 * batch, straight from physical bytes (section 4.1.1 reads them back).  Node 0
 * is the root, nodes 1..|I| are I in order, and the entry at position j < len-1
 * of tuple i of D makes the next node, whose parent is D_i[j] and whose key is
 * the first pair of D_i[j+1]'s sequence; depth is the sequence length.  The
 * first pair of a node and its depth are found by pointer jumping along parents.
 *   blobs    device bytes holding the batches' blobs; batch b is bytes
 *            blob_off[b] .. blob_off[b+1]-1 (blob_off: host, n_batches+1 entries,
 *            non-decreasing)
 *   node_off host, n_batches+1 entries: batch b's nodes are output entries
 *            node_off[b] .. node_off[b+1]-1 (toc_phys_info_get's n_nodes each)
 *   max_rows the most tuples of any batch (at most 16384; sizes LDS)
 *   n_cols   columns of the matrix the bytes encode: a column of I at or above it
 *            makes the batch malformed (TOC_CPRIME_COLUMN), so no later step
 *            indexes W or w past n_cols with it
 *   parent, col, val, depth  device outputs, one entry per node in paper
 *            numbering: the root has parent 0xFFFFFFFF, col 0xFFFFFFFF, val +0.0,
 *            depth 0; nodes 1..|I| have parent 0
 *   status   device int32 per batch: 0, or TOC_CPRIME_* below when the blob is
 *            malformed (the batch's outputs are then unspecified; nothing outside
 *            its blob and node range is touched)
 *   ws       device workspace of toc_cprime_workspace_size bytes
 * Asynchronous on stream; blob_off and node_off are copied before returning.
 * Checks the host arrays and sizes (TOC_EINVAL, TOC_ESIZE).                  */
#define TOC_CPRIME_LAYOUT 1       /* headers, widths or sizes do not hold         */
#define TOC_CPRIME_VALUE_INDEX 2  /* a value index is not below the unique count  */
#define TOC_CPRIME_STARTS 3       /* tuple starts not non-decreasing from 0 to |D| */
#define TOC_CPRIME_CODE 4         /* a code names no node existing at that point  */
#define TOC_CPRIME_NODES 5        /* the node count differs from node_off's span  */
#define TOC_CPRIME_ROWS 6         /* more tuples than max_rows                    */
#define TOC_CPRIME_COLUMN 10      /* a column of I is not below n_cols            */
toc_status toc_cprime_build(const void *blobs, const int64_t *blob_off, const int64_t *node_off,
                            int64_t n_batches, int32_t max_rows, int32_t n_cols, uint32_t *parent,
                            uint32_t *col, float *val, uint32_t *depth, int32_t *status, void *ws,
                            size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * Encoding on the device.  The logical encoding of Algorithm 1 (section 3.1)
 * after the sparse encoding (section 3), for many mini-batches held in one
 * concatenated CSR in device memory, each batch with its own prefix tree: the
 * result is the (I, D) that toc_encode gives for the same batch, node for node.
 * ------------------------------------------------------------------------- */

/* Workspace bytes of toc_encode_device for n_batches batches of at most max_nnz
 * entries each (max_nnz <= 2^30, else TOC_EUNSUPPORTED): one hash table of
 * 16-byte slots (a power of two of them, at least 1.5 max_nnz + 1 and 64) for
 * each of up to 1024 batches in phase I and for each of up to 16384 batches in
 * phase II, each phase capped near 8 GiB, plus 8 (n_batches + 1) bytes. */
toc_status toc_encode_device_workspace_size(int64_t n_batches, int64_t max_nnz, size_t *bytes);

/* Algorithm 1 on the device: phase I numbers the distinct pairs of a batch in
 * order of first appearance (one workgroup per batch), phase II encodes its
 * tuples by greedy longest matches, growing the tree (one lane per batch, the
 * tree's child links in a hash table in the workspace).
 *   n_rows   host int32[n_batches]: batch b owns the n_rows[b] rows after those
 *            of batches 0..b-1
 *   rowptr   device int64[sum(n_rows) + 1], non-decreasing; entry e (rowptr[0]
 *            <= e < rowptr[0] + nnz) is col[e - rowptr[0]], val[e - rowptr[0]]
 *   col, val device int32 / float[nnz]; the same rules as toc_encode: columns in
 *            [0, n_cols) strictly increasing inside a row, values finite; entries
 *            equal to zero (either sign) are dropped
 *   max_nnz  the most entries of any batch (sizes the workspace)
 * Outputs (device, caller-owned).  Batch b's entries occupy indexes
 * s_b = rowptr[r_b] - rowptr[0] onwards, r_b its first row; its slot there holds:
 *   I_col, I_val  int32 / float[nnz]: I (nodes 1..|I| of Algorithm 1, in order)
 *            at s_b .. s_b + |I| - 1
 *   D_codes  uint32[nnz]: D's codes of all the batch's tuples, in paper
 *            numbering, at s_b .. s_b + |D| - 1 (the rest of the slot is
 *            overwritten with unspecified values)
 *   D_rowptr int64[sum(n_rows) + n_batches]: at r_b + b, the batch's n_rows[b]+1
 *            offsets of its tuples into its D (starting at 0)
 *   counts   int64[4 n_batches]: |I|, |D|, the node count of the tree with its
 *            root (1 + |I| + sum over tuples of (codes - 1)), nonzero entries
 *   status   int32[n_batches]: 0, or TOC_ENCDEV_* below (then the batch's counts
 *            are 0 and its outputs unspecified; nothing outside its slot is
 *            written)
 *   ws       device workspace of toc_encode_device_workspace_size bytes
 * Asynchronous on stream (n_rows is copied before returning).  TOC_EINVAL for
 * NULL or negative arguments, TOC_ESIZE for a small workspace, TOC_EUNSUPPORTED
 * for max_nnz above 2^30 or 2^32-1 batches or more.  Not reentrant on one
 * workspace: calls that share a workspace must be ordered on one stream.      */
#define TOC_ENCDEV_ROWPTR 1   /* rowptr decreases at or inside the batch, or leaves
                                 [rowptr[0], rowptr[0] + nnz]                     */
#define TOC_ENCDEV_SIZE 2     /* more entries than max_nnz                        */
#define TOC_ENCDEV_COLUMN 3   /* a column out of range or not increasing in a row */
#define TOC_ENCDEV_VALUE 4    /* a value is NaN or infinite                       */
toc_status toc_encode_device(int64_t n_batches, const int32_t *n_rows, int32_t n_cols,
                             const int64_t *rowptr, const int32_t *col, const float *val,
                             int64_t nnz, int64_t max_nnz, int32_t *I_col, float *I_val,
                             uint32_t *D_codes, int64_t *D_rowptr, int64_t *counts,
                             int32_t *status, void *ws, size_t ws_bytes, void *stream);

/* Workspace bytes of toc_level_build for n_batches batches and n_nodes nodes in
 * total. */
toc_status toc_level_workspace_size(int64_t n_batches, int64_t n_nodes, size_t *bytes);

/* The live codes of each batch in level order, on the device, from the tree of
 * toc_cprime_build and the D of the same blobs: the codes D references and all
 * their ancestors (the only codes the operations of section 4 touch), stably
 * sorted by (depth, paper index), so that every parent precedes its children
 * (all the forward scan of Algorithm 4 and the backward scan of Algorithm 5
 * need); parents and D renumbered to that order.
 *   blobs, blob_off, node_off  as for toc_cprime_build (the same launch's)
 *   d_off    host, n_batches+1 entries: batch b's D is entries d_off[b] ..
 *            d_off[b+1]-1 of l_D (toc_phys_info_get's n_codes each)
 *   max_levels  deepest level kept, 1..4096 (sizes LDS and `level`)
 *   cprime_status, parent, col, val, depth  toc_cprime_build's outputs
 * Outputs (device, caller-owned):
 *   l_parent, l_col, l_val, l_depth  at node_off[b] onwards, one entry per live
 *            code in level order (parent as a level-order index, 0xFFFFFFFF at
 *            depth 1); the rest of the batch's node range is left alone
 *   level    uint32 (max_levels+1) per batch: level[d] = live codes of depth <= d
 *   l_D      D renumbered
 *   counts   int64 2 per batch: live codes, deepest live depth
 *   status   int32 per batch: 0, the batch's nonzero cprime status, TOC_CPRIME_*
 *            for a blob that does not hold, or TOC_LEVEL_* below
 * Asynchronous on stream; the offsets are copied before returning.  Needs
 * 36 (max_levels + 1) + ceil(nodes / 32) * 4 bytes of LDS for the batch with the
 * most nodes, at most 160 KiB (TOC_EUNSUPPORTED beyond).                     */
#define TOC_LEVEL_D 7             /* the blob's |D| differs from d_off's span       */
#define TOC_LEVEL_DEPTH 8         /* a live code deeper than max_levels            */
toc_status toc_level_build(const void *blobs, const int64_t *blob_off, const int64_t *node_off,
                           const int64_t *d_off, int64_t n_batches, int32_t max_levels,
                           const int32_t *cprime_status, const uint32_t *parent,
                           const uint32_t *col, const float *val, const uint32_t *depth,
                           uint32_t *l_parent, uint32_t *l_col, float *l_val, uint32_t *l_depth,
                           uint32_t *level, uint32_t *l_D, int64_t *counts, int32_t *status,
                           void *ws, size_t ws_bytes, void *stream);

/* A.w for k = 1 (Theorem 1) straight from the output of toc_level_build, so that
 * the whole path from physical bytes to a product runs on the device: per batch,
 * H over the live codes level by level in LDS (parents first), then each tuple's
 * sum of H over its renumbered codes (tuple starts read from the blob).
 *   blobs, blob_off, node_off, d_off, max_levels  as for toc_level_build
 *   row_off  host, n_batches+1 entries: batch b's tuples are rows row_off[b] ..
 *            row_off[b+1]-1 of r
 *   n_cols   entries of w; a batch with a key column at or above it gets
 *            TOC_CPRIME_COLUMN and w is never read past n_cols
 *   max_live the most live codes of a batch (4 max_live bytes of LDS, at most
 *            160 KiB, else TOC_EUNSUPPORTED; a batch above it gets TOC_LEVEL_LIVE)
 *   level_status, counts, level, l_parent, l_col, l_val, l_D  toc_level_build's
 *   w        device float[n_cols];  r  device float per row (output)
 *   status   device int32 per batch: 0, level_status when nonzero,
 *            TOC_LEVEL_D when the blob's tuples or |D| differ from the offsets, or
 *            TOC_CPRIME_COLUMN (then r's rows of the batch are not written)
 *   ws       device workspace of at least 32 (n_batches + 1) bytes
 * Asynchronous on stream; the offsets are copied before returning.          */
#define TOC_LEVEL_LIVE 9          /* more live codes than max_live                 */
toc_status toc_level_right_mul(const void *blobs, const int64_t *blob_off, const int64_t *node_off,
                               const int64_t *d_off, const int64_t *row_off, int64_t n_batches,
                               int32_t n_cols, int32_t max_levels, int64_t max_live,
                               const int32_t *level_status,
                               const int64_t *counts, const uint32_t *level,
                               const uint32_t *l_parent, const uint32_t *l_col, const float *l_val,
                               const uint32_t *l_D, const float *w, float *r, int32_t *status,
                               void *ws, size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * The upload image built on the device from physical bytes, so that only the
 * compressed bytes of section 3.2 cross from the host.  Per batch, C' is built as
 * by toc_cprime_build (Algorithm 2 over the integers read back as in section
 * 4.1.1), its live codes are put in level order (parents first, as the scans of
 * Algorithms 4 and 5 need) and the arrays the operations read are derived from it
 * (toc_dev_layout_get lists them).  The image equals the one toc_upload builds on
 * the host from the same batches (flags 0), word for word, so every operation gives
 * the same results, bit for bit, on either.  Two steps: toc_ingest_plan counts what
 * the layout needs (a census on the device, read back) and gives the image size;
 * toc_ingest_build writes the image into a caller buffer of that size.  Batches go
 * through the workspace in ranges that fit it.  Needs codes to occur at most once
 * in a tuple (true of every encoding of Algorithm 1: a code's sequence begins at a
 * column, and a tuple holds each column once).
 * ------------------------------------------------------------------------- */
#define TOC_INGEST_CHANGED 11     /* the bytes differ from those the plan counted  */

/* Workspace bytes for the batches described by info (toc_phys_info_get of each
 * blob, n_batches entries): *bytes to take all batches in one range, *min_bytes
 * (when not NULL) the least that takes the largest batch alone.  TOC_EINVAL for
 * counts out of range or a column of I at or above n_cols, TOC_EUNSUPPORTED for a
 * batch of more than 16384 tuples. */
toc_status toc_ingest_workspace_size(const toc_phys_info *info, int64_t n_batches, int32_t n_cols,
                                     size_t *bytes, size_t *min_bytes);

/* Reads the blobs on the device and plans the image.
 *   blobs     device bytes; batch b's blob is bytes blob_off[b] .. blob_off[b+1]-1
 *             (blob_off: host, n_batches + 1 entries, non-decreasing)
 *   info      host, the toc_phys_info of each blob (its node and code counts size
 *             the workspace ranges)
 *   n_cols    columns of the encoded matrix
 *   ws        device workspace (at least toc_ingest_workspace_size's *min_bytes)
 * Synchronises `stream`.  On success *dev is a planned image (operations on it
 * fail until toc_ingest_build) and *image_bytes the bytes it needs; free it with
 * toc_dev_free.  TOC_EINVAL names the first batch whose blob is malformed (the
 * status toc_cprime_build would give it), TOC_ESIZE a workspace below the need of
 * one batch. */
toc_status toc_ingest_plan(const void *blobs, const int64_t *blob_off, const toc_phys_info *info,
                           int64_t n_batches, int32_t n_cols, void *ws, size_t ws_bytes,
                           void *stream, size_t *image_bytes, toc_dev **dev);

/* Builds the planned image into buf (device memory of at least *image_bytes from
 * the plan) from the same blobs; afterwards dev is an ordinary device image bound
 * to buf on the current device.  Synchronises `stream`.  TOC_EINVAL for a dev that
 * is not planned-and-unbuilt, or for blobs that differ from those planned (the
 * batch is named; dev stays unbuilt), TOC_ESIZE for a small buf or workspace. */
toc_status toc_ingest_build(toc_dev *dev, const void *blobs, const int64_t *blob_off, void *buf,
                            size_t bytes, void *ws, size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------------------
 * Mini-batch gradient descent (section 2.1): h <- h - lr / |B| * sum over the
 * tuples (x, y) of batch B of d loss(h, x, y) / d h, for the linear models of
 * Table 1, whose loss depends on h through r = x^T h: the batch gradient is
 * A^T g with g_i = d loss / d r at r_i = (A h)_i, so a step is the right
 * product (Theorem 1), g, the left product (Theorem 2) and the update.
 * ------------------------------------------------------------------------- */
#define TOC_MGD_LINEAR 0     /* 1/2 (y - r)^2, linear regression                    */
#define TOC_MGD_LOGISTIC 1   /* log(1 + exp(-y r)), y in {-1, +1}                   */
#define TOC_MGD_HINGE 2      /* max(0, 1 - y r), y in {-1, +1}; subgradient 0 at 1  */

/* Runs the steps of batches b0 .. b0+n_batches-1 of an uploaded image in order,
 * in one launch of one workgroup (each step reads the model the previous step
 * wrote; a batch without tuples changes nothing).
 *   y  device float per row of the image (all batches' rows, stacked)
 *   h  device float[n_cols], the model, updated in place
 * Needs 4 (max rows + max stored codes of a batch) bytes of LDS, at most 160 KiB
 * (TOC_EUNSUPPORTED beyond).  Asynchronous on stream.  TOC_EINVAL for a batch
 * range outside the image, an unknown loss, a learning rate that is not finite
 * or an image in host memory.                                                  */
toc_status toc_mgd_epoch(const toc_dev *dev, int64_t b0, int64_t n_batches, int32_t loss,
                         float lr, const float *y, float *h, void *stream);

/* Device workspace bytes toc_mgd_epoch_split needs for the image in *bytes: one
 * float per row of its largest batch (a step's loss derivatives g).
 * TOC_EINVAL for NULL arguments.                                                */
toc_status toc_mgd_workspace_size(const toc_dev *dev, size_t *bytes);

/* The steps of toc_mgd_epoch (section 2.1: the right product of Theorem 1, g,
 * the left product of Theorem 2, the update) with each step split over many
 * workgroups: two launches per step on stream, in batch order.  The first sums
 * each tuple's r = x^T h over the pairs of its codes and writes g_i = d loss / d r
 * to ws; the second forms each tree code's sum of g (its own tuples, then its
 * children's sums) and, column by column over the batch's used columns, the
 * gradient (val * g over the column's leaf occurrences, val * sum over its tree
 * codes) and h_j -= lr / |B| * gradient.  y, h, loss, lr and the errors as for
 * toc_mgd_epoch; ws is caller-owned device memory of at least the bytes
 * toc_mgd_workspace_size gives (TOC_EINVAL if NULL, TOC_ESIZE if smaller), which
 * calls on other streams must not share while this call runs.  Needs
 * 4 (max rows + max tree codes of a batch + 1) bytes of LDS, at most 160 KiB
 * (TOC_EUNSUPPORTED beyond).  The sums run in a fixed order: one call over many
 * batches equals one call per batch, bit for bit (the order differs from
 * toc_mgd_epoch's, so the two agree within rounding, not bit for bit).          */
toc_status toc_mgd_epoch_split(const toc_dev *dev, int64_t b0, int64_t n_batches, int32_t loss,
                               float lr, const float *y, float *h, void *ws, size_t ws_bytes,
                               void *stream);

/* ---------------------------------------------------------------------------
 * Mini-batch gradient descent for the neural network of section 5.1 (Table 1's
 * NN row, whose matrix operations are A.M and M.A): layers m -> h1 -> h2 ->
 * n_out with sigmoid hidden units and a bias in every layer, a softmax output
 * (n_out >= 2, labels 0..n_out-1) or one sigmoid output (n_out = 1, labels 0/1),
 * cross-entropy loss; a step moves every parameter by -lr times the gradient of
 * the batch's mean loss (section 2.1).  The first layer runs on the compressed
 * batch: Z1 = A W1 + b1 by Theorem 1 and the gradient A^T dZ1 by Theorem 2.
 * ------------------------------------------------------------------------- */

/* Workspace bytes of toc_mlp_epoch: 4 (most rows of a batch) (2 h1 + 2 h2 +
 * n_out) (each part rounded up to 4 floats), plus, when 16 bytes per code exceed
 * 160 KiB of LDS (those table rows are then kept in the workspace), 32 h1 per
 * tree code of the batch with the most and 4 h1 ceil(max rows / 64) per deep
 * code of the batch with the most. */
toc_status toc_mlp_workspace_size(const toc_dev *dev, int32_t h1, int32_t h2, int32_t n_out,
                                  size_t *bytes);

/* Runs the steps of batches b0 .. b0+n_batches-1 of an uploaded image in order
 * (three launches per step on stream; a batch without tuples changes nothing).
 *   W1 [m x h1], b1 [h1], W2 [h1 x h2], b2 [h2], W3 [h2 x n_out], b3 [n_out]:
 *            device float, row-major, updated in place; W1 and b1 16-byte aligned
 *   labels   device int32 per row of the image (all batches' rows, stacked); a
 *            label outside the classes matches none (its target is all zeros)
 *   ws       device workspace of toc_mlp_workspace_size bytes, 16-byte aligned
 * h1 must be a multiple of 4 in 4..4096 (TOC_EUNSUPPORTED otherwise), h2 and
 * n_out in 1..4096.  TOC_EINVAL for
 * a batch range outside the image, NULL or misaligned pointers, a learning rate
 * that is not finite or an image in host memory; TOC_ESIZE for a small
 * workspace.  Asynchronous on stream.                                        */
toc_status toc_mlp_epoch(const toc_dev *dev, int64_t b0, int64_t n_batches, int32_t h1,
                         int32_t h2, int32_t n_out, float *W1, float *b1, float *W2, float *b2,
                         float *W3, float *b3, const int32_t *labels, float lr, void *ws,
                         size_t ws_bytes, void *stream);

/* Message for the last non-OK status returned on this thread. */
const char *toc_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* TOC_H */
