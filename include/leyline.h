/*
 * leyline.h -- C ABI of the MI355X (gfx950) KV-cache splice library (libleyline.so).
 *
 * The library implements the data-parallel hot path of a policy-driven KV-cache edit:
 * a directive replaces the cached token span [span_start, span_end) of a sequence by a
 * replacement ("stub") of stub_len tokens whose K/V the caller has already computed at their
 * final positions (the directive 4-tuple and its positional contract: paper Sec. 3.1; the
 * tensor effect of each step: appendix "Kernel specification: tensors and composition").
 * Every cached token downstream of the span moves by Delta = stub_len - (span_end - span_start);
 * its rotary key band is re-anchored with the closed-form rotation k' = R(Delta) k
 * (paper Eq. "rotate", Sec. 3.2), while non-rotary data (MLA latent c_kv / K_nope, GQA V) is
 * moved bit-for-bit.  Several non-overlapping directives per call are applied left to right with
 * a running (cumulative) shift of either sign; overlapping spans are rejected (appendix "Kernel
 * specification", multiple directives).  RoPE pairs are interleaved (dims 2i, 2i+1) or half-split
 * (dims i, i+d/2) per plane (Sec. 3.3 "RoPE pairing convention").  Rotation arithmetic is fp32
 * with cos/sin of the exact integer shift times theta_i evaluated in fp64 once per call and
 * directive; results are rounded to nearest-even into the storage dtype (Sec. 4.1 "bf16 K-storage
 * precision floor").
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Return value: LEYLINE_OK (0) or a negative LEYLINE_E_* code; leyline_strerror() names it.
 * - All arguments are validated before anything is enqueued: a call that returns an error has
 *   not touched device memory (the per-call all-or-none rule).  A failure reported by the HIP
 *   runtime after the first enqueue (LEYLINE_E_HIP) cannot be rolled back.
 * - "device" pointers are HIP device memory owned by the caller; "host" pointers are ordinary
 *   host memory read (or written) only during the call.  The library never allocates or frees
 *   device memory and keeps no state between calls; it is re-entrant.
 * - stream is a hipStream_t passed as void* (NULL = the default stream).  Device work is
 *   asynchronous on it; host outputs are complete when the call returns.  The caller orders the
 *   call against kernels that read the cache.
 * - Element offsets and strides are counted in elements of the cache dtype.  Every device base
 *   pointer must be 16-byte aligned and every row, stride, head and rotary band must span a
 *   multiple of 16 bytes (rows are moved as 16-byte vectors); otherwise LEYLINE_E_INVAL.
 */
#ifndef LEYLINE_H
#define LEYLINE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LEYLINE_ABI_VERSION 3
#define LEYLINE_MAX_PLANES 4

enum {
    LEYLINE_OK = 0,
    LEYLINE_E_INVAL = -1,     /* null pointer, bad descriptor, misaligned layout             */
    LEYLINE_E_RANGE = -2,     /* span outside [0, seq_len], seq index out of range            */
    LEYLINE_E_ORDER = -3,     /* directives not sorted by (seq, span_start)                   */
    LEYLINE_E_OVERLAP = -4,   /* two spans of one sequence overlap                            */
    LEYLINE_E_CAPACITY = -5,  /* new length > capacity, too few free pages, output too small  */
    LEYLINE_E_MODE = -6,      /* a FORGET directive that is not the last of its sequence, or  */
                              /* that carries a replacement                                   */
    LEYLINE_E_WORKSPACE = -7, /* workspace missing or smaller than the query reported         */
    LEYLINE_E_HIP = -8        /* the HIP runtime reported an error while enqueueing           */
};

/* Storage dtype of the whole cache (all planes). */
enum { LEYLINE_BF16 = 0, LEYLINE_F32 = 1 };

/* RoPE pairing of a plane's rotary bands (Sec. 3.3): interleaved pairs dims (2i, 2i+1) of the
 * band; NEOX (half-split) pairs dims (i, i + rot_dim/2). */
enum { LEYLINE_ROPE_INTERLEAVED = 0, LEYLINE_ROPE_NEOX = 1 };

/* Directive mode (Sec. 3.1, "The FORGET mode").  AMORTIZE is the splice: replacement written,
 * downstream rows moved and re-anchored.  FORGET asks for true forgetting, which the serving stack
 * implements as a prefix-trimmed re-prefill: on the cache, the sequence is cut at the FORGET
 * span's start (after the effect of the earlier directives) and nothing is moved or rotated; the
 * caller then re-prefills from there.  A FORGET directive must be the last directive of its
 * sequence and carry no replacement (stub_len = 0), else LEYLINE_E_MODE. */
enum { LEYLINE_AMORTIZE = 0, LEYLINE_FORGET = 1 };

/* Flags of the paged calls.  COPY_ON_WRITE: no old page is written.  A page whose rows all come
 * from one old page with a nonzero whole-page shift is assembled into a fresh page instead of
 * being re-used with its rotary bands rotated in place, so pages shared with other sequences (a
 * radix prefix cache) keep their contents; the rotated KV goes to fresh pages, as the Role A/B
 * integration of Sec. 3.3 writes it to fresh destination slots. */
enum { LEYLINE_PAGED_COPY_ON_WRITE = 1 };

/* Device-side status bits a kernel may OR into the optional device_status word. */
enum {
    LEYLINE_STATUS_BAD_PAGE = 1,     /* a block-table or free-list entry was outside [0, capacity) */
    LEYLINE_STATUS_BAD_ROW = 2,      /* a row index given to leyline_rotate_delta was out of range  */
    LEYLINE_STATUS_TILE_TIMEOUT = 4  /* an ordered tile of a contiguous splice gave up waiting for  */
                                     /* a tile it depends on (see leyline_splice_contig)           */
};

/*
 * One tensor family stored per token and layer.  MLA caches have one plane (row = latent c_kv
 * followed by K_pe); GQA caches have a K plane (rotated over whole heads) and a V plane (moved
 * only).  Row r of layer l starts at element
 *     contiguous cache: base + l*layer_stride + r*token_stride
 *     paged cache:      base + l*layer_stride + page*page_stride + (r % page_size)*token_stride
 * A row holds row_elems elements; head h < n_heads starts at h*head_stride within the row and
 * carries rot_dim rotary elements starting at rot_offset within the head (rot_dim = 0: the plane
 * is moved only).  Frequencies are theta_i = rope_base^(-2i/rot_dim) (RoFormer), or inv_freq[i]
 * when inv_freq (host, rot_dim/2 doubles) is non-NULL.
 */
typedef struct leyline_plane {
    void* base;             /* device */
    int64_t layer_stride;   /* elements between layers */
    int64_t token_stride;   /* elements between consecutive rows (within a page when paged) */
    int64_t page_stride;    /* elements between physical pages (paged only; ignored otherwise) */
    int32_t row_elems;
    int32_t n_heads;        /* >= 1 when rot_dim > 0 */
    int32_t head_stride;
    int32_t rot_offset;
    int32_t rot_dim;        /* even; 0 = no rotary band */
    int32_t rope_style;     /* LEYLINE_ROPE_* */
    double rope_base;
    const double* inv_freq; /* host, nullable */
} leyline_plane;

typedef struct leyline_cache {
    int32_t dtype;          /* LEYLINE_BF16 or LEYLINE_F32 */
    int32_t n_layers;       /* >= 1 */
    int32_t n_planes;       /* 1 .. LEYLINE_MAX_PLANES */
    int32_t page_size;      /* 0: contiguous cache; > 0: tokens per page */
    int64_t capacity;       /* contiguous: rows allocated per layer; paged: physical pages in the pool */
    leyline_plane planes[LEYLINE_MAX_PLANES];
} leyline_cache;

/*
 * A directive D = (span_start, span_end, R, mode) of Sec. 3.1, in the pre-call coordinates of
 * sequence `seq` (0 for a contiguous cache).  stub[p] is the replacement's K/V for plane p:
 * device memory, dense [n_layers][stub_len][row_elems] in the cache dtype, already RoPE'd at its
 * final positions [span_start + running_shift, ... + stub_len); it is copied verbatim and never
 * rotated.  stub[p] may be NULL only when stub_len == 0.  An empty span (pure insertion) and an
 * empty stub (pure deletion) are both valid.
 */
typedef struct leyline_directive {
    int32_t seq;
    int32_t mode;           /* LEYLINE_AMORTIZE or LEYLINE_FORGET */
    int64_t span_start;
    int64_t span_end;
    int64_t stub_len;
    const void* stub[LEYLINE_MAX_PLANES];
} leyline_directive;

/* Human-readable name of a return code (static storage). */
const char* leyline_strerror(int code);

/* LEYLINE_ABI_VERSION of the loaded library. */
int leyline_abi_version(void);

/* Precision of the loaded library's rotation arithmetic: 32 or 64.  libleyline.so (32) takes
 * cos/sin rounded to fp32 and computes each rotated pair in fp32 (the paper's policy, Sec. 4.1
 * "bf16 K-storage precision floor"), then rounds once to the storage dtype.  libleyline_exact.so
 * (64) takes fp64 cos/sin and computes in fp64, then rounds once to the storage dtype, so stored
 * values are the correctly rounded exact rotation (bit-identical to a float64 reference up to
 * fp64 rounding).  Both export the same entry points. */
int leyline_pair_bits(void);

/* The HIP runtime's description of the error behind the last LEYLINE_E_HIP returned on the
 * calling thread ("no error" if there was none).  Static storage. */
const char* leyline_last_hip_error(void);

/*
 * Host-only check of a contiguous splice: validates exactly as leyline_splice_contig does and
 * reports (host outputs, each nullable) the new length, the number of kernel launches the splice
 * will enqueue, how many of them are ordered-tile launches, and the device workspace it needs in
 * bytes (0 when the splice runs without ordered tiles).  Enqueues nothing.
 */
int leyline_contig_query(const leyline_cache* cache, int64_t seq_len,
                         const leyline_directive* dirs, int32_t n_dirs,
                         int64_t* new_len_out, int32_t* n_launches_out,
                         int32_t* n_tile_launches_out, int64_t* workspace_bytes_out);

/*
 * Contiguous in-place splice of one sequence (all layers and planes).
 *
 * cache->page_size must be 0; rows [0, seq_len) hold the sequence, capacity rows are allocated.
 * dirs: host array of n_dirs >= 0 directives (seq = 0), sorted by span_start, non-overlapping
 * (adjacent spans are allowed).  After the call, rows [0, *new_len_out) hold the spliced sequence:
 * prefix rows untouched, each stub at its new position, each downstream row at its old position
 * plus the running shift with its rotary bands rotated by that shift.  Rows [new_len, max(seq_len,
 * new_len)) are left unspecified.  Source and destination ranges overlap; the library orders the
 * moves so that every row is read before it is overwritten.  When every shift is large against
 * its segment the moves run as rounds (independent launches); otherwise the whole call (moves and
 * stub copies of every directive) runs as ordered tiles, normally in a single launch, whose
 * workgroups coordinate through counters and flags in the workspace.
 *
 * workspace: device memory, 256-byte aligned, at least the size leyline_contig_query reports
 * (NULL allowed when that size is 0); it holds the tiles' ticket counters and flags and the
 * call's cos/sin table.  The call writes it on `stream` before use; reuse it only after the
 * stream has passed this call, and do not share one workspace between calls that may run at the
 * same time.
 * device_status: device int32, nullable.  A tile waits for the tiles whose source rows its
 * destination overlaps; each wait is bounded (a few hundred milliseconds at least, where a
 * correct schedule waits microseconds).  A tile that gives up ORs LEYLINE_STATUS_TILE_TIMEOUT
 * into *device_status and stores nothing, so every workgroup still exits; the cache content is
 * then unspecified.  This can only follow from a schedule fault or from two calls running at the
 * same time on one workspace.
 * Enqueues kernels only (all parameters travel as kernel arguments; the workspace is cleared and
 * filled by a kernel), so the call may be captured into a HIP graph; each replay repeats the same
 * splice.
 * Errors: E_INVAL, E_RANGE, E_ORDER, E_OVERLAP, E_CAPACITY (new length > capacity), E_MODE,
 * E_WORKSPACE (missing, misaligned or too small), E_HIP.
 */
int leyline_splice_contig(const leyline_cache* cache, int64_t seq_len,
                          const leyline_directive* dirs, int32_t n_dirs,
                          int64_t* new_len_out, int32_t* device_status,
                          void* workspace, int64_t workspace_bytes, void* stream);

/* Bytes of the library's fixed per-GPU scratch array used by leyline_splice_contig_noalloc. */
#define LEYLINE_SCRATCH_BYTES (1 << 20)

/*
 * leyline_splice_contig without any device allocation, for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc).
 *
 * Same splice, arguments, validation, kernels and results as leyline_splice_contig, but the
 * workspace is a fixed array of LEYLINE_SCRATCH_BYTES bytes in device memory that the library
 * holds on each GPU it runs on until the process ends (located on the first call on a device).
 * The call uses the calling thread's current device; a non-NULL stream must belong to it
 * (E_INVAL otherwise).  A splice whose ordered tiles need more workspace than
 * LEYLINE_SCRATCH_BYTES returns LEYLINE_E_WORKSPACE before anything is enqueued (1 MiB holds
 * the counters and flags of, e.g., a small-shift splice of a 61-layer MLA cache of about 480K
 * tokens); use leyline_splice_contig with a caller workspace for those.  The call makes no
 * device allocation or free (no hipMalloc / hipFree, no allocating library routine) and clears
 * the counters and flags it needs with a kernel at its start.  Every call on one GPU shares that
 * GPU's array: calls that may overlap in time on one GPU (other streams, other threads) race and
 * must be ordered by the caller.
 */
int leyline_splice_contig_noalloc(const leyline_cache* cache, int64_t seq_len,
                                  const leyline_directive* dirs, int32_t n_dirs,
                                  int64_t* new_len_out, int32_t* device_status, void* stream);

/*
 * Sizes of a paged splice, computed on the host from lengths and directives alone.
 *
 * cache: the paged cache the splice will run on (its plane layout sizes the cos/sin tables).
 * seq_lens: host [n_seqs]; bt_stride: row length of the block tables; flags: LEYLINE_PAGED_*
 * (as for the splice); dirs: host, sorted by
 * (seq, span_start).  Outputs (host, each nullable): new_seq_lens[n_seqs]; *n_fresh_needed =
 * fresh pages the call will consume; *n_freed = pages the call will drop from block tables;
 * *workspace_bytes = device workspace the call needs.
 * Errors: as leyline_splice_paged's validation (E_CAPACITY when a new table exceeds bt_stride).
 */
int leyline_paged_query(const leyline_cache* cache, int32_t n_seqs, const int32_t* seq_lens,
                        int32_t bt_stride, const leyline_directive* dirs, int32_t n_dirs,
                        uint32_t flags, int32_t* new_seq_lens, int32_t* n_fresh_needed,
                        int32_t* n_freed, int64_t* workspace_bytes);

/* Page kinds of a paged plan. */
enum { LEYLINE_PAGE_IDENTITY = 0, LEYLINE_PAGE_REMAP = 1, LEYLINE_PAGE_ASSEMBLE = 2, LEYLINE_PAGE_NONE = -1 };

/*
 * Symbolic page plan (host only), for schedulers and tests.  For new logical page k of sequence
 * b (k < ceil(new_len/page_size)):
 *   IDENTITY: every row comes from the same position of old logical page k, shift 0;
 *             the physical page is kept and not touched.
 *   REMAP:    every row comes from old logical page src at the same in-page offset with one
 *             nonzero shift (a multiple of page_size); the physical page is re-used and only its
 *             rotary bands are rotated in place.
 *   ASSEMBLE: the rows are gathered into fresh page number src (fresh pages are numbered in
 *             ascending (b, k) order and taken from free_pages in that order).
 * Old logical pages referenced by neither IDENTITY nor REMAP are freed, listed in ascending
 * (b, old page) order.  The paper describes no paging; this rule is the library's own.
 *
 * kind_out, src_out: host [n_seqs][bt_stride] (LEYLINE_PAGE_NONE / -1 past the new length);
 * freed_seq_out, freed_page_out: host [freed_cap].  E_CAPACITY when bt_stride or freed_cap is
 * too small.
 */
int leyline_paged_plan(int32_t page_size, int32_t n_seqs, const int32_t* seq_lens,
                       const leyline_directive* dirs, int32_t n_dirs, uint32_t flags,
                       int32_t bt_stride,
                       int32_t* kind_out, int32_t* src_out,
                       int32_t* freed_seq_out, int32_t* freed_page_out, int32_t freed_cap);

/*
 * Paged splice of a batch of sequences (all layers and planes), following the page plan above.
 *
 * cache->page_size > 0, cache->capacity = physical pages in the pool.
 * seq_lens: host [n_seqs].  block_table_in / block_table_out: device int32 [n_seqs][bt_stride]
 * (bt_stride >= 0; 0 only when every sequence is and stays empty, and then the tables may be null);
 * on completion block_table_out holds every sequence's new table and -1 past its last page.
 * The old and new block tables, free_pages [n_free], freed_pages_out [freed_cap], the workspace
 * [workspace_bytes] and device_status [1] are read and written by the same launch: no two of
 * them may share a byte (E_INVAL).  free_pages: device int32 [n_free], consumed from index 0 by ASSEMBLE pages.
 * freed_pages_out: device int32 [freed_cap], receives the dropped physical pages.
 * Host outputs (nullable): new_seq_lens_out[n_seqs], *n_fresh_used_out, *n_freed_out.
 * device_status: device int32, nullable; kernels OR LEYLINE_STATUS_* bits into it when a page
 * index read from device memory is outside [0, capacity) (that row is then skipped).
 * workspace: device, 256-byte aligned, >= the size leyline_paged_query reports.  It receives the
 * plan (runs of pages, per-sequence and per-directive tables and cos/sin; plans of at most 2560
 * bytes travel in the kernel arguments instead, larger ones are uploaded with an asynchronous
 * copy on `stream`) and, when the call assembles more than 1024 rows, the row table a kernel of
 * this call writes from it (24 bytes per row of every ASSEMBLE page, 4 bytes per fresh page);
 * when some plane rotates at least 1 KiB per row and at least 64 pages are re-used, the REMAP
 * pages resolved and sorted by physical page (16 bytes per REMAP page);
 * reuse it only after the stream has passed this call.  Any page_size whose rows keep the
 * 16-byte alignment is accepted.  A call with a plan of at most 2560 bytes enqueues kernels only
 * (and, assembling at most 1024 rows, a single one); an uploaded plan comes from host memory the
 * call owns only while it runs: do not capture such a call into a HIP graph.
 *
 * flags: 0, or LEYLINE_PAGED_COPY_ON_WRITE (no REMAP pages: no old page is written).
 * Ownership: only ASSEMBLE pages (fresh) and REMAP pages (rotary bands, in place) are written.
 * Pages holding the rows of a REMAP page must not be shared with another sequence (pass
 * LEYLINE_PAGED_COPY_ON_WRITE when they may be).  Freed pages
 * are not written; the caller may recycle them once the stream has passed this call.
 * Errors: as leyline_splice_contig, plus E_CAPACITY (too few free pages, freed_cap or bt_stride
 * too small) and E_WORKSPACE.
 */
int leyline_splice_paged(const leyline_cache* cache, int32_t n_seqs, const int32_t* seq_lens,
                         const int32_t* block_table_in, int32_t* block_table_out, int32_t bt_stride,
                         const leyline_directive* dirs, int32_t n_dirs, uint32_t flags,
                         const int32_t* free_pages, int32_t n_free,
                         int32_t* freed_pages_out, int32_t freed_cap,
                         int32_t* new_seq_lens_out, int32_t* n_fresh_used_out, int32_t* n_freed_out,
                         int32_t* device_status,
                         void* workspace, int64_t workspace_bytes, void* stream);

/*
 * In-place re-anchoring without movement: every rotary band of the given rows, in every layer,
 * becomes R(delta) times itself (Eq. "rotate").  Non-rotary elements are not touched.
 *
 * Rows are physical: contiguous cache -> row index r < capacity; paged cache -> page*page_size +
 * offset with page < capacity.  rows: device int64 [n_rows] (nullable: then rows row0 ..
 * row0+n_rows-1).  Listed rows must be distinct.  device_status as above (out-of-range listed
 * rows are skipped and flagged with LEYLINE_STATUS_BAD_ROW).
 * Errors: E_INVAL (also: a paged pool of 2^31 or more rows, or more than 2^31 band chunks in one
 * plane's call), E_RANGE (row0 range outside the cache), E_HIP.
 */
int leyline_rotate_delta(const leyline_cache* cache, int64_t delta,
                         const int64_t* rows, int64_t row0, int64_t n_rows,
                         int32_t* device_status, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* LEYLINE_H */
