/*
 * pulse.h -- C ABI of libpulse, the MI355X (gfx950) PULSE patch codec.
 *
 * The library implements the data-parallel hot path of compute-visible
 * sparsification (arXiv 2602.03839):
 *   - the BF16 view of FP32 master weights (Sec. 3 "Sparsity metric"),
 *   - the sparse value patch of PULSESync: encode (Sec. 4.2, Alg. 1 Encode;
 *     App. H.5, Alg. 3) and apply (Alg. 1 Decode; App. H.5, Alg. 4),
 *   - PULSELoCo's error-feedback sparsification of FP32 pseudo-gradients
 *     and its outer step, SparseSync's average plus outer Nesterov momentum
 *     (Sec. 4.3, Alg. 2),
 *   - the delta-varint index stream (App. H.2, App. F.3) and the weight hash
 *     a receiver checks after applying a patch (App. J.4).
 *
 * Conventions for every entry point:
 *   - Pointers are DEVICE pointers (HIP device memory of the current device)
 *     unless the argument says "host".  BF16 values travel as uint16_t bit
 *     patterns.
 *   - `stream` is a hipStream_t passed as void* (NULL = the default stream).
 *     Work is enqueued on it and the call returns without synchronising; the
 *     caller owns every buffer and keeps it alive until the stream has run
 *     the work.  The library allocates no device memory.
 *   - Return value: PULSE_OK, or a negative pulse_status for an argument error
 *     found on the host (nothing is enqueued then) or a failed launch.
 *     pulse_strerror() names it; pulse_last_error() gives the detail message
 *     of the calling thread's last failure.
 *   - n == 0 (or an empty batch) enqueues nothing that changes outputs.
 *
 * Patch layout (Sec. 4.2 "Encoding and decoding": store index and new value,
 * not a difference; App. H.2: indices ascending): struct-of-arrays
 * `uint32_t idx[capacity]` + value array, entries in ascending index order,
 * tensors in the order given.  Index of element i of a tensor = index_base + i,
 * so a whole model below 2^32 parameters can use one flat index space
 * (index_base = offset of the tensor), and larger models use per-tensor local
 * indices (index_base = 0) with per-tensor segment offsets (seg_begin).
 *
 * Running count: `count` is a device uint64.  On entry it holds the number of
 * entries already in the patch (the append position); the kernel adds the
 * number of entries this call selects, also those that did not fit.  Entries
 * whose position is >= capacity are not written; the caller detects overflow
 * as *count > capacity after synchronising.
 *
 * Workspace: encode and sparsify need `pulse_workspace_bytes()` bytes of
 * device memory, 256-byte aligned, ZERO-FILLED ONCE before its first use and
 * then reused unchanged by every call (the kernels leave it valid for the next
 * call).  Calls that share a workspace must be ordered on one stream; give
 * concurrent streams separate workspaces.  A call that faulted leaves it
 * undefined: zero it again.
 *
 * Workspace misuse is detected, not hidden: a workspace that was not
 * zero-filled can make a tile wait for a predecessor that never publishes.
 * The kernels then stop waiting (within a fraction of a second), treat the
 * missing tiles as empty -- so the patch, counts and segment offsets of that
 * call are wrong -- and raise a flag in the workspace (64-bit word 16, byte
 * offset 128).  The flag stays raised, and every later call on that workspace
 * stops waiting at once, until the caller zero-fills the workspace again.
 * pulse_workspace_status() reads it.
 */
#ifndef PULSE_H
#define PULSE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum pulse_status {
    PULSE_OK = 0,
    PULSE_EINVAL = -1, /* NULL required pointer, bad size, workspace too small */
    PULSE_ERANGE = -2, /* index_base + n > 2^32 */
    PULSE_EALIGN = -3, /* a dense stream pointer is not 16-byte aligned */
    PULSE_EHIP = -4,   /* the HIP runtime rejected a launch */
    PULSE_ESTATE = -5  /* the workspace flag is raised: a look-back gave up */
} pulse_status;

/* Size in bytes of the workspace that encode and sparsify calls use. */
size_t pulse_workspace_bytes(void);

/*
 * pulse_workspace_status -- whether every call on `workspace` since it was
 * last zero-filled found all its predecessors' status words (see "Workspace
 * misuse" above).  Synchronises `stream` (the stream the calls were ordered
 * on), then reads the workspace's flag with a device-to-host copy.
 *   workspace        as passed to the calls; workspace_bytes its size.
 * Returns PULSE_OK when the flag is clear, PULSE_ESTATE when it is raised
 * (the results of the calls since the last zero-fill are unreliable; zero the
 * workspace before reusing it), PULSE_EINVAL / PULSE_EALIGN for a bad
 * workspace argument and PULSE_EHIP if the copy fails.
 */
int pulse_workspace_status(const void *workspace, size_t workspace_bytes, void *stream);

/* Human-readable name of a pulse_status value (static string). */
const char *pulse_strerror(int status);

/* Detail message of the calling thread's last failed call ("" if none). */
const char *pulse_last_error(void);

/*
 * pulse_cast_bf16 -- the BF16 view of an FP32 tensor (Sec. 3 "Sparsity
 * metric": the dtype of the next forward pass), dst[i] = bf16(src[i]),
 * round to nearest, ties to even (App. A.2, App. D).  A NaN becomes a quiet
 * NaN with the same sign and leading payload bits.  Used for the first
 * snapshot / full anchor of a chain.
 *   src  FP32 [n], 16-byte aligned.      dst  BF16 bits [n], 16-byte aligned.
 */
int pulse_cast_bf16(const float *src, uint16_t *dst, uint64_t n, void *stream);

/*
 * pulse_encode -- PULSESync encode of one tensor (Sec. 4.2, Alg. 1 Encode;
 * App. H.5, Alg. 3).  I = { i : bf16(w_new[i]) != snap[i] } compared bitwise
 * (Sec. 3: equality is bitwise, so +0 != -0), V = bf16(w_new)[I]; entry k of
 * this tensor's part of the patch is written at position (*count on entry) + k
 * as idx = index_base + i, val = bf16(w_new[i]).
 *   w_new       FP32 master after the step [n], 16-byte aligned.
 *   snap        previous BF16 snapshot [n], 16-byte aligned; read only, unless
 *               it is also `refresh`.
 *   n           elements; index_base + n <= 2^32 (else PULSE_ERANGE).
 *   idx, val    patch arrays with room for `capacity` entries.
 *   count       device uint64, in: append position, out: += entries selected.
 *   refresh     NULL, or BF16 [n] that receives bf16(w_new[i]) for every
 *               EMITTED entry (position < capacity); may equal `snap`, which
 *               advances the snapshot in place (App. H.3).
 *   workspace   pulse_workspace_bytes() bytes, see above.
 */
int pulse_encode(const float *w_new, const uint16_t *snap, uint64_t n,
                 uint32_t *idx, uint16_t *val, uint64_t capacity, uint64_t *count,
                 uint32_t index_base, uint16_t *refresh,
                 void *workspace, size_t workspace_bytes, void *stream);

/*
 * Flags of a batched encode tensor.
 *
 * PULSE_REFRESH_MIRRORS_SNAP: the caller guarantees that refresh[i] == snap[i]
 * (same bits) at every position i that this call does not select, which holds
 * when `refresh` is W_{t-1}, the copy Alg. 1 Decode starts from
 * (W_t <- W_{t-1}; W_t[I] <- V).  The result is then the same as without the
 * flag, but the kernel may rewrite unselected elements with their own value:
 * it writes whole aligned 128-byte runs of `refresh` that contain an emitted
 * change, instead of one 2-byte write per change.  `refresh` must then be
 * 16-byte aligned (else PULSE_EALIGN).  A refresh that IS the snapshot
 * (refresh == snap) is treated this way without the flag.  If the guarantee
 * does not hold, unselected elements of such runs take snap's value.
 */
#define PULSE_REFRESH_MIRRORS_SNAP 1u

/* One tensor of a batched encode (fields as in pulse_encode). */
typedef struct pulse_encode_tensor {
    const float *w_new;
    const uint16_t *snap;
    uint16_t *refresh; /* may be NULL */
    uint64_t n;
    uint32_t index_base;
    uint32_t flags;    /* 0 or PULSE_REFRESH_MIRRORS_SNAP */
} pulse_encode_tensor;

/*
 * pulse_encode_batch -- Alg. 3's loop over parameter tensors in one pass: the
 * tensors' patches are appended one after another, in the order given, to one
 * patch.  Equivalent to calling pulse_encode on each tensor in order.
 *   tensors     HOST array [ntensors]; read during the call only.
 *   seg_begin   NULL, or device uint64 [ntensors]: position in the patch where
 *               tensor t's entries begin (the end of tensor t is seg_begin[t+1],
 *               and *count for the last one).  Values may exceed capacity.
 */
int pulse_encode_batch(const pulse_encode_tensor *tensors, uint32_t ntensors,
                       uint32_t *idx, uint16_t *val, uint64_t capacity, uint64_t *count,
                       uint64_t *seg_begin, void *workspace, size_t workspace_bytes,
                       void *stream);

/*
 * pulse_encode_batch_noalloc -- pulse_encode_batch without a workspace
 * argument, for callers that cannot allocate device memory: code being
 * captured into a HIP graph, tight serving loops, harnesses that forbid
 * hipMalloc.  The call allocates nothing (no hipMalloc/hipFree, no
 * allocating library routine); its scratch is a 524,800-byte array inside
 * the library (pulse_workspace_bytes()), one per GPU, held from the first
 * call on that GPU until the process ends.  Each call first clears the
 * scratch with a small fill kernel on `stream`, then runs exactly the
 * launches of pulse_encode_batch, so results are identical to it.
 *   Arguments and errors: as pulse_encode_batch, less the workspace.  A call
 *   that would need more scratch than the library holds is rejected with
 *   PULSE_EINVAL (none does today: the scratch does not grow with n); a
 *   device index above 63 is rejected with PULSE_EINVAL.
 *   Concurrency: every call on one GPU shares that GPU's scratch, so calls
 *   that overlap on one GPU (different streams, or threads) race and give
 *   wrong patches; order them on one stream.
 */
int pulse_encode_batch_noalloc(const pulse_encode_tensor *tensors, uint32_t ntensors,
                               uint32_t *idx, uint16_t *val, uint64_t capacity,
                               uint64_t *count, uint64_t *seg_begin, void *stream);

/*
 * pulse_apply -- PULSESync decode of one tensor (Sec. 4.2, Alg. 1 Decode;
 * App. H.5, Alg. 4): dst[idx[k] - index_base] = val[k] for k in
 * [*begin, min(*end, capacity)).  A direct copy of bit patterns, no
 * arithmetic; dst is not read.  Indices must be unique (encode's are); entries
 * whose index is outside [index_base, index_base + n) are skipped and, if
 * `rejected` is not NULL, counted into the device uint64 *rejected.
 *   dst       BF16 [n] receiving the patch in place (App. H.3).
 *   begin/end device uint64 positions (e.g. a saved count and encode's count),
 *             so no host synchronisation is needed between encode and apply.
 */
int pulse_apply(uint16_t *dst, uint64_t n, const uint32_t *idx, const uint16_t *val,
                uint64_t capacity, const uint64_t *begin, const uint64_t *end,
                uint32_t index_base, uint64_t *rejected, void *stream);

/* One tensor of a batched apply. */
typedef struct pulse_apply_tensor {
    uint16_t *dst;
    uint64_t n;
    uint32_t index_base;
} pulse_apply_tensor;

/*
 * pulse_apply_batch -- Alg. 4's loop over tensors: tensor t takes the entries
 * [seg_begin[t], seg_begin[t+1]) (the last one up to *end), clipped to
 * capacity, as produced by pulse_encode_batch.
 *   tensors    HOST array [ntensors].
 *   seg_begin  device uint64 [ntensors], non-decreasing.
 */
int pulse_apply_batch(const pulse_apply_tensor *tensors, uint32_t ntensors,
                      const uint32_t *idx, const uint16_t *val, uint64_t capacity,
                      const uint64_t *seg_begin, const uint64_t *end, uint64_t *rejected,
                      void *stream);

/*
 * pulse_loco_sparsify -- PULSELoCo sparsification with error feedback
 * (Sec. 4.3, Alg. 2): a = fl32(delta[i] + residual[i]) (s = Delta + e), then
 *   theta == NULL: selected iff |a| >= tau (threshold form);
 *   theta != NULL: selected iff bf16(theta[i]) != bf16(fl32(theta[i] - a)),
 *                  the compute-visibility gate G_BF16(theta, s) of Sec. 4.1
 *                  (tau is ignored).
 * A selected entry at position < capacity is emitted as (index_base + i, a)
 * and its residual becomes +0 (e[I] <- 0); every other entry -- not selected,
 * or selected but beyond capacity, hence not sent -- keeps residual = a
 * (e[not I] <- s).  NaN is never selected by the threshold form.
 *   delta, residual (in/out), theta: FP32 [n], 16-byte aligned.
 *   idx, val   FP32 patch with room for `capacity` entries.
 *   workspace  at least pulse_workspace_bytes() bytes, see above.  With a
 *              larger one (pulse_loco_workspace_bytes) the threshold form
 *              runs in two passes, with the same results.
 */
int pulse_loco_sparsify(const float *delta, float *residual, uint64_t n, float tau,
                        const float *theta, uint32_t *idx, float *val, uint64_t capacity,
                        uint64_t *count, uint32_t index_base,
                        void *workspace, size_t workspace_bytes, void *stream);

/* One tensor of a batched sparsify. */
typedef struct pulse_loco_tensor {
    const float *delta;
    float *residual;
    const float *theta; /* may be NULL: threshold form */
    uint64_t n;
    uint32_t index_base;
} pulse_loco_tensor;

/*
 * pulse_loco_workspace_bytes -- size of a workspace with which a threshold-
 * form sparsify call (no theta; pulse_loco_sparsify[_batch]) over tensors of
 * at most n elements in all runs entirely in its two-pass form.  The first
 * pass streams Delta and e as many short-lived blocks in address order (the
 * fastest way this chip streams a read-modify-write), staging each 1,024-
 * element tile's selected entries in the workspace; the second writes them
 * to the patch in index order.  The results -- patch, count, seg_begin,
 * residual -- are bit-identical to the one-pass form's.
 * The part of the workspace past pulse_workspace_bytes() holds the staging
 * area and needs no initialisation; the first pulse_workspace_bytes() keep
 * the rules above (zero-filled once), so one workspace may serve every call
 * ordered on a stream.  A call whose launch (<= 64 tensors) needs more
 * staging than the workspace holds runs that launch in one pass; the gate
 * forms always run in one pass.  About 1 byte of workspace per element.
 */
size_t pulse_loco_workspace_bytes(uint64_t n);

/* pulse_loco_sparsify over tensors in order, appended to one patch (see pulse_encode_batch). */
int pulse_loco_sparsify_batch(const pulse_loco_tensor *tensors, uint32_t ntensors, float tau,
                              uint32_t *idx, float *val, uint64_t capacity, uint64_t *count,
                              uint64_t *seg_begin, void *workspace, size_t workspace_bytes,
                              void *stream);

/*
 * One worker's sparse FP32 list for the outer step, as pulse_loco_sparsify
 * writes it: entries in strictly ascending index order within each tensor,
 * indices of the form index_base + i.
 *   idx, val    device arrays; entries at positions >= capacity are ignored.
 *   seg_begin   device uint64 [ntensors]: position of each tensor's first entry.
 *   end         device uint64: one past the last tensor's last entry (e.g.
 *               the sparsifier's count).
 */
typedef struct pulse_sparse_list {
    const uint32_t *idx;
    const float *val;
    uint64_t capacity;
    const uint64_t *seg_begin;
    const uint64_t *end;
} pulse_sparse_list;

#define PULSE_MAX_LISTS 8 /* workers per call */

/* One tensor of the outer step. */
typedef struct pulse_outer_tensor {
    float *theta;    /* FP32 [n], in/out, 16-byte aligned */
    float *momentum; /* FP32 [n], in/out, 16-byte aligned (zero before the first round) */
    uint64_t n;
    uint32_t index_base;
} pulse_outer_tensor;

/*
 * pulse_outer_step_batch -- PULSELoCo's outer update (Sec. 4.3, Alg. 2: the
 * SparseSync line and the two lines after it), per tensor:
 *   g_i = (sum over workers r, in list order, of r's value at index i) / R,
 *         a worker without an entry at i counting as zero; g = 0 if R == 0;
 *   m_i     <- mu * m_i + g_i
 *   theta_i <- theta_i - alpha * (mu * m_i + g_i)    (m_i the new momentum)
 * every operation rounded to FP32 on its own (no fused multiply-add).  The
 * paper uses mu = 0.9, alpha = 0.7.  g is formed on the fly from the sorted
 * lists; nothing is allocated.  Entries whose index lies outside the tensor
 * are ignored; unsorted lists give an undefined result.
 *   tensors   HOST array [ntensors]; lists HOST array [nlists], nlists <= PULSE_MAX_LISTS.
 */
int pulse_outer_step_batch(const pulse_outer_tensor *tensors, uint32_t ntensors,
                           const pulse_sparse_list *lists, uint32_t nlists,
                           float mu, float alpha, void *stream);

/* pulse_outer_step_batch for one tensor; each list's seg_begin points to the
 * position of the tensor's first entry and `end` one past its last. */
int pulse_outer_step(float *theta, float *momentum, uint64_t n, uint32_t index_base,
                     const pulse_sparse_list *lists, uint32_t nlists,
                     float mu, float alpha, void *stream);

/*
 * pulse_varint_encode -- the delta-varint index stream of a sorted patch
 * (App. H.2 "Index Encoding": sort, first index as it is, then differences;
 * App. F.3 "Sparse stream format": indices delta-encoded and varint-packed).
 * Per segment (one per tensor) the first index is written as it is and every
 * later one as its difference from the previous, each as an unsigned varint
 * (7-bit groups, least significant first, 0x80 on every byte but the last of
 * a number).  Segments follow each other in order; values are not part of the
 * stream (they stay in the patch's value array).
 *   idx         device uint32 [capacity], indices ascending within each segment.
 *   end         device uint64: the number of entries (e.g. encode's count);
 *               only entries below min(*end, capacity) are read.
 *   seg_begin   NULL (one segment) or device uint64 [nseg], non-decreasing:
 *               the entry where each segment starts (encode's seg_begin).
 *               Entry 0 always starts a segment.
 *   out         device bytes, `out_capacity` of them; bytes past it are not
 *               written, *total_bytes still receives the full length.
 *   seg_bytes   NULL or device uint64 [nseg]: the byte where each segment's
 *               numbers start (an empty segment: where the next one starts).
 *   total_bytes device uint64: the stream's length.
 *   workspace   the encode/sparsify workspace (same rules; may be shared on
 *               one stream).
 * The stream is at most nnz + (N - nnz)/127 bytes for nnz entries out of N
 * positions (App. F.3 accounting).
 */
int pulse_varint_encode(const uint32_t *idx, uint64_t capacity, const uint64_t *end,
                        const uint64_t *seg_begin, uint32_t nseg,
                        uint8_t *out, uint64_t out_capacity,
                        uint64_t *seg_bytes, uint64_t *total_bytes,
                        void *workspace, size_t workspace_bytes, void *stream);

/*
 * pulse_varint_decode -- indices back from a delta-varint stream (Alg. 1
 * Decode's DeltaDecode step).
 *   in          device bytes [in_capacity], 16-byte aligned (EALIGN), with
 *               in_capacity < 2^40 (EINVAL); *nbytes (device uint64) of them
 *               form the stream.  A stream cut inside a number drops it; a
 *               number of more than five bytes (not a uint32 varint) decodes
 *               to an unspecified value.
 *   seg_begin   NULL (one segment) or device uint64 [nseg]: the entry where
 *               each segment starts (container metadata sent with the stream).
 *   idx         device uint32 [capacity] receiving the indices; entries past
 *               capacity are not written.
 *   count       device uint64: the number of entries in the stream.
 *   workspace   as for encode.  The decode keeps its per-tile sums in the
 *               workspace's status ring and leaves them zero, so the workspace
 *               stays valid for the other ordered kernels on the same stream.
 * Five launches (count, offsets, segment-start tiles, carries, write): the
 * stream is read twice and the indices written once; no block waits on
 * another.
 */
int pulse_varint_decode(const uint8_t *in, uint64_t in_capacity, const uint64_t *nbytes,
                        const uint64_t *seg_begin, uint32_t nseg,
                        uint32_t *idx, uint64_t capacity, uint64_t *count,
                        void *workspace, size_t workspace_bytes, void *stream);

/*
 * pulse_coo_encode -- the 2-D COO delta downcast of a sorted patch's indices
 * (App. H.2 step 4: downcast the index types, uint8 row deltas and uint16
 * column deltas; App. H.4.1 "Type downscaling").  Segment s (one tensor,
 * row-major with cols[s] columns, 1 <= cols[s] <= 65535) is written as
 *   first[s]      its first index as it is (App. H.2 step 2; 0 if empty),
 *   then one (drow uint8, dcol uint16) pair per later entry:
 *     same row as the previous entry:  (0, column - previous column)
 *     dr rows further down:            (dr, column + 1)     for dr <= 255
 *     dr > 255:                        (255, 0) escapes, each 255 rows down
 *                                      with no entry, ahead of the pair of the
 *                                      remaining 1..255 rows.
 *   No entry yields (255, 0).  Pairs of segment s start at seg_pairs[s];
 *   *total_pairs receives the stream's length; pairs at or past out_capacity
 *   are not written.  idx, capacity, end and the workspace follow
 *   pulse_varint_encode; seg_begin[0] should be 0 (earlier entries count as
 *   segment 0).  cols, first and seg_pairs are device arrays of nseg >= 1
 *   elements.  A stream of P pairs takes 3 P bytes plus 4 bytes per segment.
 *   Indices must ascend within each segment; an entry below the one before
 *   it gets one unspecified pair (the stream is then not decodable), and no
 *   access leaves the buffers.
 */
int pulse_coo_encode(const uint32_t *idx, uint64_t capacity, const uint64_t *end,
                     const uint64_t *seg_begin, uint32_t nseg, const uint32_t *cols,
                     uint32_t *first, uint8_t *drow, uint16_t *dcol, uint64_t out_capacity,
                     uint64_t *seg_pairs, uint64_t *total_pairs,
                     void *workspace, size_t workspace_bytes, void *stream);

/*
 * pulse_coo_decode -- the indices back from a 2-D COO delta stream (Alg. 1
 * Decode's Upcast and DeltaDecode steps for pulse_coo_encode's format).
 *   drow, dcol    device [pair_capacity], both 16-byte aligned (EALIGN),
 *                 pair_capacity < 2^40 (EINVAL); *npairs (device) of them
 *                 form the stream.
 *   seg_begin     device [nseg]: the entry where each segment starts; *nent
 *                 (device) the number of entries (container metadata sent
 *                 with the stream, as encode's seg_begin and count).
 *   seg_pairs, first, cols   as pulse_coo_encode wrote / read them.
 *   idx           device uint32 [capacity]: entry k of the patch at idx[k];
 *                 entries at or past capacity are not written.
 * Each pair acts on the (row, column) of the entry before it: (0, gap) moves
 * the column, (dr, c + 1) moves dr rows down to column c, an escape 255 rows
 * down.  These maps compose, so three launches (fold each tile's pairs, scan
 * the tile folds, write) give every pair its row, column and escape count since
 * its segment's start, and its entry lands at seg_begin[s] + 1 + (pairs of s
 * before it) - (escapes of s before it).  The library allocates nothing: the
 * per-tile folds live in the workspace's status ring and are left zero.  A
 * stream that encode did not write decodes to unspecified indices but no
 * access leaves the buffers.
 */
int pulse_coo_decode(const uint8_t *drow, const uint16_t *dcol, uint64_t pair_capacity,
                     const uint64_t *npairs, const uint64_t *seg_begin, const uint64_t *seg_pairs,
                     uint32_t nseg, const uint32_t *cols, const uint32_t *first,
                     const uint64_t *nent, uint32_t *idx, uint64_t capacity,
                     void *workspace, size_t workspace_bytes, void *stream);

/*
 * Receivers that compute in a precision below BF16 (App. D): the compute view
 * cast_D of the FP32 masters, the patch of the values whose view changes
 * (Alg. 1 with D in place of BF16), and its apply on the receiver's D copy.
 *   PULSE_DTYPE_FP8_E4M3  OCP FP8 E4M3 (bias 7, no infinity, largest 448).
 *       A tensor carries an FP32 scale: the receiver computes with
 *       fl32(w * inv_scale), rounded to the nearest code (ties to the even
 *       code), saturating to +-448 (also for +-inf); NaN -> 0x7F with its sign.
 *       One uint8 code per value.
 *   PULSE_DTYPE_MXFP4     OCP MXFP4: blocks of 32 consecutive values of a
 *       tensor (the last may be shorter) share one E8M0 scale byte E + 127,
 *       E = clamp(exponent field of the block's largest |w| - 129, -127, 127)
 *       (= floor(log2 max|w|) - 2 for a normal maximum); each value is the
 *       E2M1 code (sign, 2 exponent bits, 1 mantissa bit) of w / 2^E, nearest
 *       with ties to the even code, saturating to +-6.  A block holding a NaN
 *       gets scale 0xFF and codes 0.  Codes are packed two per byte, the
 *       even-indexed value in the low nibble: (n + 1) / 2 code bytes and
 *       (n + 31) / 32 scale bytes per tensor.  A value's compute view is the
 *       pair (its block's scale, its code); a patch entry's value is
 *       (scale << 8) | code as uint16, so a scale change re-sends its block.
 */
#define PULSE_DTYPE_FP8_E4M3 1
#define PULSE_DTYPE_MXFP4 2

/* Dense D view of one tensor: FP8 codes[n] (8-byte aligned), or MXFP4 packed
 * codes (4-byte aligned) and scales. `src` 16-byte aligned; inv_scale is
 * used by FP8 only; scales may be NULL for FP8. */
int pulse_cast_lowp(int dtype, const float *src, uint64_t n, float inv_scale,
                    uint8_t *codes, uint8_t *scales, void *stream);

typedef struct pulse_lowp_tensor {
    const float *w_new;          /* FP32 masters, 16-byte aligned */
    const uint8_t *snap;         /* the receiver's D view: FP8 codes (8-byte aligned) or
                                    MXFP4 packed codes (4-byte aligned) */
    const uint8_t *snap_scales;  /* MXFP4 scale bytes; unused for FP8 */
    uint64_t n;
    uint32_t index_base;
    float inv_scale;             /* FP8 only */
} pulse_lowp_tensor;

/*
 * pulse_encode_lowp_batch -- Alg. 1 Encode for a receiver computing in D:
 * every value whose D view differs bitwise from the snapshot's is emitted as
 * (index_base + i, value) in index order, tensors in the order given; value =
 * the FP8 code (val: uint8[capacity]) or (scale << 8) | code (val:
 * uint16[capacity], 2-byte aligned).  idx, count, seg_begin, capacity and
 * the workspace follow pulse_encode_batch.  The snapshot is not refreshed:
 * the receiver's copy is brought up to date by pulse_apply_lowp_batch.
 */
int pulse_encode_lowp_batch(int dtype, const pulse_lowp_tensor *tensors, uint32_t ntensors,
                            uint32_t *idx, void *val, uint64_t capacity, uint64_t *count,
                            uint64_t *seg_begin, void *workspace, size_t workspace_bytes,
                            void *stream);

typedef struct pulse_lowp_apply_tensor {
    uint8_t *codes;   /* FP8 codes or MXFP4 packed codes */
    uint8_t *scales;  /* MXFP4 scale bytes; unused for FP8 */
    uint64_t n;
    uint32_t index_base;
} pulse_lowp_apply_tensor;

/*
 * pulse_apply_lowp_batch -- Alg. 1 Decode on a D copy: entry k of tensor t's
 * segment [seg_begin[t], next start or *end) writes its code to value
 * idx[k] - index_base (MXFP4: its nibble, and its scale to the value's
 * block).  Indices must be unique and ascending within a segment (as encode
 * writes them); entries outside the tensor are counted in *rejected.
 */
int pulse_apply_lowp_batch(int dtype, const pulse_lowp_apply_tensor *tensors, uint32_t ntensors,
                           const uint32_t *idx, const void *val, uint64_t capacity,
                           const uint64_t *seg_begin, const uint64_t *end,
                           uint64_t *rejected, void *stream);

/*
 * pulse_loco_sparsify_lowp_batch -- Alg. 2's selection with the gate of a
 * receiver that computes in D (App. D: G_D(theta, s) = {i : cast_D(theta_i) !=
 * cast_D(theta_i - s_i)}): a = fl32(delta + e) is selected iff
 * cast_D(theta) and cast_D(fl32(theta - a)) differ at i -- for FP8 the codes
 * of fl32(theta * inv_scales[t]) and fl32((theta - a) * inv_scales[t]), for
 * MXFP4 the (block scale, code) pairs, each vector's blocks scaled by their
 * own maximum.  Every tensor needs theta; inv_scales (host array, one per
 * tensor) is read for FP8 only.  Emission, capacity, residual, counts and the
 * workspace are those of pulse_loco_sparsify_batch.
 */
int pulse_loco_sparsify_lowp_batch(int dtype, const pulse_loco_tensor *tensors,
                                   const float *inv_scales, uint32_t ntensors,
                                   uint32_t *idx, float *val, uint64_t capacity, uint64_t *count,
                                   uint64_t *seg_begin, void *workspace, size_t workspace_bytes,
                                   void *stream);

/*
 * Weight hash (App. J.4 "Weight-level integrity", "Deterministic hashing"):
 * a SHA-256 digest of the BF16 bit patterns of all tensors, concatenated in
 * the order given, that the sender publishes with each patch and the receiver
 * recomputes over the weights it rebuilt.
 *
 * The message is the tensors' bytes as they sit in memory (each value's two
 * bytes, low byte first).  One SHA-256 over it cannot be split across a GPU,
 * so the digest is a tree of SHA-256 (FIPS 180-4): the message is cut into
 * leaves of PULSE_HASH_LEAF_BYTES bytes (the last may be shorter) and the
 * leaves are combined by the Merkle Tree Hash of RFC 6962, Sec. 2.1:
 *   leaf digest  SHA-256(0x00 || leaf bytes)
 *   node digest  SHA-256(0x01 || left digest || right digest), the left
 *                subtree holding the largest power of two of leaves below the
 *                count;
 *   no leaves    SHA-256 of the empty message.
 * The digest depends only on the concatenated bytes, not on how they are
 * split into tensors.  A message of at most one leaf hashes to
 * SHA-256(0x00 || message).
 */
#define PULSE_HASH_LEAF_BYTES 16384

typedef struct pulse_hash_tensor {
    const uint16_t *data; /* device; 4-byte aligned; may be NULL when n == 0 */
    uint64_t n;           /* BF16 values */
} pulse_hash_tensor;

/* Number of leaves of a message of `total_values` BF16 values. */
uint64_t pulse_hash_leaf_count(uint64_t total_values);

/* Workspace bytes pulse_hash_tree needs for `ntensors` tensors holding
 * `total_values` values together (not the encode workspace; it needs no
 * zero-filling). */
size_t pulse_hash_workspace_bytes(uint32_t ntensors, uint64_t total_values);

/*
 * pulse_hash_tree -- the weight hash of `ntensors` tensors (host array).
 *   leaf_digests  device, 32 * pulse_hash_leaf_count(total) bytes, 4-byte
 *                 aligned: every leaf's digest (FIPS byte order), kept so that
 *                 a mismatch can be narrowed to 16 KiB chunks. May be NULL
 *                 only when there are no values.
 *   root          device, 32 bytes, 4-byte aligned: the digest.
 *   workspace     device, 256-byte aligned, pulse_hash_workspace_bytes() bytes.
 * Errors: EINVAL (NULL pointer, workspace too small), EALIGN, EHIP.
 */
int pulse_hash_tree(const pulse_hash_tensor *tensors, uint32_t ntensors,
                    uint8_t *leaf_digests, uint8_t *root,
                    void *workspace, size_t workspace_bytes, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* PULSE_H */
