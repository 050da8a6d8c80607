/*
 * bsr.h -- C ABI of the Bounded-State Restoration (BSR) restore path on one
 * MI355X (gfx950) GPU.
 *
 * BSR (arxiv 2608.17826) restores one rank's externally retained KV state
 * into an engine's paged KV cache through a reusable local staging window of
 * at most W chunks.  It has three phases (§3 "Protocol: Probe, Install,
 * Commit"):
 *   probe   -- find the complete reusable prefix without staging it (§3
 *              "Probe globally"; §4 "LMCache changes", probe-only mode);
 *   install -- move the confirmed prefix window by window through W staging
 *              slots into the destination blocks (§2 "Bounded installation",
 *              Eqs. 3-4; §3 "Install locally"; §4 windowed retrieve);
 *   commit  -- expose the prefix only if every group is valid, otherwise
 *              invalidate the whole advertised prefix (§3 Eq. 6, Prop. 2;
 *              §4 "vLLM failure integration").
 *
 * Conventions
 *   - Every function returns an int status: BSR_OK (0) or a negative
 *     BSR_E_* code.  No exception crosses the ABI.  bsr_last_error() returns
 *     a thread-local message describing the last failure on that thread.
 *   - Every out-parameter is caller-allocated.  Pointers marked "device" are
 *     HIP device pointers on the context's device; all others are host
 *     pointers.  Streams are hipStream_t handles passed as void*.
 *   - Sizes are in bytes unless named *_tokens, *_chunks or *_blocks.
 *   - One context serves one GPU rank.  Every call is thread safe: calls on
 *     one context are serialised by its mutex, except that bind (reading the
 *     block tables back), commit and teardown do not hold it while they wait
 *     for the device, so other requests' calls go on meanwhile; device work
 *     of different requests overlaps on their streams.  Destroy a context
 *     only once every other call on it has returned.  By default one request at a time
 *     may be bound (the bounded-retrieve lock of §3 "Install locally");
 *     a global admission budget B (bsr_config.staging_budget_bytes, §7) lets
 *     several be bound while their staging rings together stay within B.
 *
 * Data layout
 *   A chunk is chunk_tokens consecutive tokens.  A group is one allocator
 *   group of the paged cache: n_tensors registered tensors sharing a block
 *   size (block_tokens) and a block table.  A record is one tensor's
 *   record_bytes for one token.
 *   - External entry of (chunk i, group g): n_tensors * chunk_tokens records,
 *     tensor-major then token-minor ([t][q][record]).
 *   - Staging slot (one chunk): group g's entry at byte offset off_g, with
 *     off_0 = 0 and off_{g+1} = off_g + align_up(payload_g, 256); the slot
 *     size is off_G (bsr_slot_bytes).  The staging ring is W slots.
 *   - Destination pool of tensor t of group g: pool_blocks blocks of
 *     block_tokens * record_bytes bytes.  Token tau lives in block
 *     block_table[tau / block_tokens] at position o = tau % block_tokens.
 *     CONTIG blocks keep records in token order (offset o*record_bytes).
 *     PLANAR blocks keep the first split_bytes of each record at
 *     o*split_bytes and the remaining bytes at
 *     block_tokens*split_bytes + o*(record_bytes - split_bytes).
 *   - Validity: one byte per pool block per group (1 = valid state).
 */
#ifndef BSR_H
#define BSR_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define BSR_ABI_VERSION 4
#define BSR_MAX_GROUPS 8
#define BSR_MAX_INSTALL_BATCH 32
#define BSR_MAX_BOUND_REQUESTS 16 /* session slots of one context */
#define BSR_STATIC_SCRATCH_BYTES (2u << 20) /* per-GPU scratch of bsr_ctx_create_static contexts */
#define BSR_NO_CHUNK 0xFFFFFFFFu

/* status codes */
#define BSR_OK 0
#define BSR_E_ARG (-1)       /* invalid argument (sizes, layout, pointers, block ids) */
#define BSR_E_STATE (-2)     /* call out of protocol order */
#define BSR_E_MISSING (-3)   /* a store entry of the window is absent */
#define BSR_E_CORRUPT (-4)   /* reserved for callers: corruption is reported through commit */
#define BSR_E_TIMEOUT (-5)   /* the window's fetch exceeded its deadline */
#define BSR_E_TRANSFER (-6)  /* a HIP transfer or launch failed */
#define BSR_E_NOMEM (-7)     /* store arena full or host/device allocation failed */
#define BSR_E_STAGING (-8)   /* staging buffer smaller than W * slot bytes, or a ring larger than B */
#define BSR_E_BUSY (-9)      /* no admission now: the lock is held, B is used up or no session slot is free */
#define BSR_E_DEVICE (-10)   /* operation needs a GPU context */
#define BSR_E_NOTFOUND (-11) /* unknown key or request */

/* failure reasons recorded in bsr_dev_status.fail */
#define BSR_FAIL_NONE 0
#define BSR_FAIL_MISSING 1
#define BSR_FAIL_CORRUPT 2
#define BSR_FAIL_TIMEOUT 3
#define BSR_FAIL_TRANSFER 4
#define BSR_FAIL_ABORT 5
#define BSR_FAIL_BLOCK_TABLE 6 /* an advertised block id lies outside its pool (BSR_FLAG_TRUSTED_TABLES) */

/* group kinds */
#define BSR_KIND_CONTIG 0
#define BSR_KIND_PLANAR 1

/* bsr_config.flags */
#define BSR_FLAG_TIME_INSTALL 1u  /* time every install launch with HIP events */
#define BSR_FLAG_TIME_STAGE 16u   /* time every staging-kernel launch with HIP events.  Each stamp on the
                                      copy stream lengthens the gap between two consecutive staging copies,
                                      which the restore then pays (0.2-0.4% of a 512K restore at W = 32,
                                      1% at W = 8) */
#define BSR_FLAG_TRUSTED_TABLES 2u /* bind does not read the block tables back, so it never waits for the
                                      compute stream (an engine's model work may be queued there); the
                                      tables are checked on the device after the begin kernel instead: an
                                      id outside [0, pool_blocks) fails the request (fail = BSR_FAIL_BLOCK_TABLE,
                                      nothing exposed; the kernels never write such an id).  The caller
                                      guarantees that no id repeats within one group's prefix (not checked) */
#define BSR_FLAG_TWO_STREAMS 8u   /* stage every request on the copy stream.  By default a request of at
                                      most 64 MiB of chunks is staged on the compute stream, so that stream
                                      order, not events between the two streams, orders its copies,
                                      installs and slot reuse */
#define BSR_FLAG_SDMA_COPIES 4u   /* stage chunks with the copy engine (hipMemcpyAsync) instead of the
                                      library's staging-copy kernel.  By default a small kernel on the copy
                                      stream reads each run of chunks from pinned host memory (the library's
                                      arena, an adopted arena that HIP reports pinned over its whole range,
                                      or the file tier's bounce buffers) into the ring; a source HIP does not
                                      report pinned is always copied by the copy engine, and so is every run
                                      staged on a copy stream while more than one request is bound */

/* fault injection (bsr_debug_inject), forced from the host */
#define BSR_INJECT_NONE 0
#define BSR_INJECT_DELAY_MS 1       /* sleep param ms before fetching chunk */
#define BSR_INJECT_TRANSFER_ERROR 2 /* treat chunk's copy submission as failed */
#define BSR_INJECT_LAUNCH_ERROR 3   /* the first install flush holding chunk reports a failed launch
                                       (nothing is launched; one shot) */

/* external tiers, in the probe's order of preference (§4 "System topology":
 * remote DRAM first, local SSD as the lower reusable tier) */
#define BSR_TIER_PINNED 0 /* the pinned-host store (bsr_store_*) */
#define BSR_TIER_FILE 1   /* the file-backed lower tier (bsr_file_tier_*) */
#define BSR_TIER_NONE 255

/* bsr_file_tier_open flags */
#define BSR_FILE_DIRECT 1u /* read chunk files with O_DIRECT (bypass the page cache) */

/* struct ids for bsr_struct_size */
#define BSR_STRUCT_LAYOUT 1
#define BSR_STRUCT_CONFIG 2
#define BSR_STRUCT_GROUP_DST 3
#define BSR_STRUCT_DEV_STATUS 4
#define BSR_STRUCT_STATS 5
#define BSR_STRUCT_ADMISSION 6

typedef struct bsr_group_desc {
  uint32_t block_tokens; /* tokens per destination block, >= 1 */
  uint32_t n_tensors;    /* registered tensors in the group, >= 1 */
  uint32_t record_bytes; /* bytes per token per tensor, multiple of 4 */
  uint32_t kind;         /* BSR_KIND_CONTIG or BSR_KIND_PLANAR */
  uint32_t split_bytes;  /* PLANAR: first-plane bytes per record, multiple of 4, < record_bytes */
} bsr_group_desc;

typedef struct bsr_layout {
  uint32_t chunk_tokens; /* tokens per chunk (the unit of W), >= 1 */
  uint32_t n_groups;     /* 1..BSR_MAX_GROUPS */
  bsr_group_desc groups[BSR_MAX_GROUPS];
} bsr_layout;

typedef struct bsr_config {
  uint32_t window_chunks;     /* W: staging slots, the restore-window size; 0 = legacy whole-plan mode
                                 (§4 "Restore-window configuration": each request's ring holds its whole
                                 plan, n_hit slots, none reused; peak staging n_hit * slot bytes, Eq. 2) */
  uint32_t install_batch;     /* chunks per install launch, 0 = automatic (W - max(1, W/8), at least 1, at
                                 most BSR_MAX_INSTALL_BATCH); <= min(W, BSR_MAX_INSTALL_BATCH).  Batches may span
                                 windows; a batch smaller than W keeps the staging copies going across windows.
                                 BSR_E_ARG when one launch of this many chunks would exceed HIP's 2^32 - 1
                                 work-items (a layout of very many small tensors): lower it */
  int32_t hip_device;         /* HIP device ordinal; -1 = host-only context (store + probe only) */
  uint32_t flags;             /* BSR_FLAG_*; unknown bits are an error */
  uint32_t window_timeout_ms; /* per-window fetch deadline, 0 = none */
  uint32_t max_bound_requests;   /* session slots: requests that may be bound at once, each with its own
                                    pre-allocated tag partials, verify words, events and status mirror.
                                    0 = automatic: 1 when staging_budget_bytes is 0, else
                                    min(BSR_MAX_BOUND_REQUESTS, B / (max(W, 1) * slot bytes)), i.e. as
                                    many as B can hold; <= BSR_MAX_BOUND_REQUESTS, and <= 1 when
                                    staging_budget_bytes is 0 */
  uint64_t staging_budget_bytes; /* B, the global admission budget (§7 "Current concurrency is
                                    conservative"): 0 keeps the bounded-retrieve lock (one bound request
                                    at a time, §3 "Install locally").  B > 0 admits a bind while the
                                    rings of every bound request plus its own
                                    (bsr_plan_staging_bytes each) stay <= B; with a bounded window B must
                                    hold at least one ring */
} bsr_config;

/* Destination of one group for one request (all pointers device, caller-owned). */
typedef struct bsr_group_dst {
  const int32_t* block_table; /* device int32[n_blocks]: physical block of the request's k-th block */
  void* const* tensor_bases;  /* device array of n_tensors device pointers, each to a pool of
                                 pool_blocks * block_tokens * record_bytes bytes, 16-byte aligned */
  uint8_t* valid;             /* device uint8[pool_blocks]: validity byte per pool block */
  uint32_t n_blocks;          /* entries in block_table; >= ceil(n_hit*chunk_tokens/block_tokens) */
  uint32_t pool_blocks;       /* blocks per pool tensor; every block id used must be < pool_blocks */
} bsr_group_dst;

/* Request status word block, device-resident and caller-allocated (64 bytes).
 * Written only by the library's kernels, in stream order on the compute
 * stream.  exposed_tokens is non-zero only after a successful commit. */
typedef struct bsr_dev_status {
  uint32_t fail;               /* BSR_FAIL_* of the first failure, 0 = none */
  uint32_t first_failed_chunk; /* chunk index of the first failure, BSR_NO_CHUNK = none */
  uint32_t q[BSR_MAX_GROUPS];  /* Eq. 6 per-group validity q_g: 1 valid, 0 invalid */
  uint64_t exposed_tokens;     /* tokens exposed as reusable (0 or n_hit*chunk_tokens) */
  uint32_t fallback;           /* 1 when the request must fall back (failed commit or invalidate) */
  uint32_t phase;              /* 1 bound, 2 committed, 3 invalidated */
  uint32_t reserved[2];
} bsr_dev_status;

/* Host-side counters of one request (bsr_stats_get, bsr_request_stats). */
typedef struct bsr_stats {
  uint64_t request_id;
  uint32_t n_hit_chunks;        /* n: prefix length bound for restore */
  uint32_t window_chunks;       /* W */
  uint32_t install_batch;       /* chunks per install launch */
  uint32_t n_windows;           /* restore_window calls accepted */
  uint32_t n_chunks_enqueued;   /* chunks whose copy and install were enqueued */
  uint32_t n_install_launches;
  uint64_t slot_bytes;             /* c: bytes of one staged chunk */
  uint64_t staging_required_bytes; /* W * slot_bytes: the ring the caller provides */
  uint64_t peak_live_staging_bytes;/* max slots holding an unreleased chunk, times slot_bytes */
  uint64_t aux_device_bytes;       /* library-owned device memory of the request's session slot, O(W)
                                      (Eq. 4 M_aux) */
  uint64_t h2d_bytes;              /* bytes enqueued host -> device */
  uint64_t installed_bytes;        /* payload bytes enqueued for installation */
  uint64_t exposed_tokens;         /* from the last commit */
  int32_t fallback;                /* from the last commit or invalidate */
  int32_t fail_reason;             /* BSR_FAIL_* from the last commit */
  uint32_t first_failed_chunk;     /* from the last commit */
  uint32_t q_mask;                 /* bit g = q_g from the last commit */
  uint64_t probe_ns;               /* host time of the last probe */
  uint64_t enqueue_ns;             /* host time spent inside restore_window calls */
  uint64_t commit_wait_ns;         /* host time commit waited for the device */
  double install_ms_total;         /* sum of install-kernel durations (BSR_FLAG_TIME_INSTALL) */
  double install_ms_max;           /* longest install launch (BSR_FLAG_TIME_INSTALL) */
  uint64_t host_bounce_bytes;      /* pinned host landing zone of the file tier (when it served chunks) */
  uint32_t file_tier_chunks;       /* chunks restored from the file tier */
  uint32_t n_stage_launches;       /* staging-copy kernel launches (0 when the copy engine staged) */
  uint64_t stage_bytes;            /* bytes those launches moved from pinned host memory */
  double stage_ms_total;           /* sum of their durations (BSR_FLAG_TIME_STAGE) */
} bsr_stats;

/* Admission state of a context (the lock or the global budget B). */
typedef struct bsr_admission {
  uint64_t staging_budget_bytes;     /* B as configured (0 = the bounded-retrieve lock) */
  uint32_t max_bound_requests;       /* session slots */
  uint32_t n_bound;                  /* requests bound now */
  uint64_t bound_staging_bytes;      /* sum of the rings of the bound requests */
  uint64_t peak_bound_staging_bytes; /* its maximum since the context was created */
  uint32_t peak_n_bound;             /* most requests bound at once */
  uint32_t n_refused;                /* binds refused with BSR_E_BUSY */
  uint64_t aux_device_bytes;         /* library-owned device memory of all session slots */
} bsr_admission;

typedef struct bsr_ctx bsr_ctx;


/* ---- library / layout ---------------------------------------------------- */

/* BSR_ABI_VERSION of the loaded library. */
int32_t bsr_abi_version(void);

/* Instrumentation: set the context's timing flags (BSR_FLAG_TIME_INSTALL,
 * BSR_FLAG_TIME_STAGE; the other config flags are kept).  A request takes
 * the flags in force when it is bound, so its counters always describe
 * the same launches.  BSR_E_ARG for any other bit. */
int bsr_set_timing(bsr_ctx* ctx, uint32_t flags);

/* sizeof of the public struct named by a BSR_STRUCT_* id, 0 if unknown
 * (lets bindings check their struct mirrors). */
uint64_t bsr_struct_size(int32_t which);

/* Thread-local message of the last failure on this thread ("" if none).
 * The pointer stays valid until the next call on this thread. */
const char* bsr_last_error(void);

/* c of §2: bytes of one staged chunk for this layout (off_G above);
 * 0 if the layout is invalid. */
uint64_t bsr_slot_bytes(const bsr_layout* layout);

/* Eq. 5 analogue M(W) = W * c: the staging ring size the caller must
 * provide.  0 if the layout is invalid or W == 0. */
uint64_t bsr_staging_bytes(const bsr_layout* layout, uint32_t window_chunks);

/* Ring bytes a request of n_hit_chunks needs on this context: W * c, or
 * n_hit_chunks * c in whole-plan mode (W = 0).  0 on a NULL context. */
uint64_t bsr_plan_staging_bytes(bsr_ctx* ctx, uint32_t n_hit_chunks);

/* Chunk keys of a token sequence (§2 restore plan; the key function is this
 * library's reading, the paper fixes none):
 *   d_i = FNV-1a-64 of the little-endian int32 tokens of chunk i,
 *   h_i = FNV-1a-64 of LE64(h_{i-1}) || LE64(d_i), h_{-1} = salt,
 * for i < floor(n_tokens / chunk_tokens); a trailing partial chunk has no
 * key.  keys_out (host, floor(n_tokens/chunk_tokens) entries) may be NULL
 * only when there are no full chunks. */
int bsr_chunk_keys(uint64_t salt, const int32_t* tokens, uint64_t n_tokens,
                   uint32_t chunk_tokens, uint64_t* keys_out);

/* ---- context --------------------------------------------------------------- */

/* Create a context for one rank.  With hip_device >= 0 the library creates
 * its HIP events and O(W) device auxiliary state on that device; with -1 only
 * the store and probe are usable.  *out is NULL on failure. */
int bsr_ctx_create(const bsr_layout* layout, const bsr_config* config, bsr_ctx** out);

/* For callers that cannot allocate device or pinned memory (code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same context as bsr_ctx_create, except that it makes no device or pinned
 * allocation.  It calls neither hipMalloc, hipHostMalloc, hipFree nor any
 * other allocating routine of HIP; it does create the context's HIP events.
 * Its one session slot's device scratch (the install kernel's tag partials
 * and the verify words) lives in a static array of
 * BSR_STATIC_SCRATCH_BYTES inside the library, one per GPU, held from the
 * first such context on that GPU until the process ends.  The status
 * mirror that commit reads back into is plain host memory of the context.
 * Requirements: hip_device >= 0, staging_budget_bytes = 0 and
 * max_bound_requests <= 1 (the bounded-retrieve lock), else BSR_E_ARG; the
 * scratch of one install launch, install_batch x (workgroups per chunk) x
 * 16 B plus 64 B of verify words, must fit the array, else BSR_E_ARG (lower
 * install_batch).  Every request of such a context on a GPU uses that GPU's
 * array, which keeps the last request's contents.  Each bind clears the
 * verify words, and each install writes every partial its verify reads.
 * Requests that overlapped on one GPU's array would race, so the library
 * allows one such context per GPU per process at a time: a second
 * bsr_ctx_create_static on the same device returns BSR_E_BUSY until the
 * first is destroyed.  Pair it with bsr_store_adopt and a caller arena,
 * because bsr_store_reserve allocates.  Destroy with bsr_ctx_destroy.  *out
 * is NULL on failure. */
int bsr_ctx_create_static(const bsr_layout* layout, const bsr_config* config, bsr_ctx** out);

/* Destroy a context: waits for outstanding device work of bound requests,
 * frees library-owned memory (arena, events, aux).  NULL is a no-op. */
int bsr_ctx_destroy(bsr_ctx* ctx);

/* ---- external tier: pinned-host store ---------------------------------------- */

/* Reserve a library-owned pinned host arena (hipHostMalloc) of at least
 * `bytes`, used for subsequent puts.  Needs a GPU context.  Once. */
int bsr_store_reserve(bsr_ctx* ctx, uint64_t bytes);

/* Use a caller-owned host arena of `bytes` (pinned by the caller for GPU
 * use; plain memory is enough for host-only contexts).  The caller keeps it
 * alive until bsr_ctx_destroy.  Once. */
int bsr_store_adopt(bsr_ctx* ctx, void* host_arena, uint64_t bytes);

/* Store one chunk under `key`: copies group_payloads[g] (payload_g bytes each,
 * [t][q][record] order) into one arena block laid out like a staging slot,
 * records a tag per group ((XOR of LE u32 words) << 32 | (sum of LE u32 words
 * mod 2^32)), and publishes one entry per (key, group).  An existing entry of
 * the key is replaced.  BSR_E_NOMEM when the arena is full. */
int bsr_store_put_chunk(bsr_ctx* ctx, uint64_t key, const void* const* group_payloads);

/* Store n chunks, as n calls of bsr_store_put_chunk would, into arena blocks
 * that are consecutive when the never-used part of the arena can hold all n
 * (else into any free blocks).  keys[i] is chunk i's key; group_payloads
 * holds n * n_groups pointers, chunk-major (chunk i, group g at
 * i * n_groups + g).  Copies and tags run on up to 8 host threads.  Chunks
 * of one prefix stored together sit back to back, as their staging slots do,
 * so a restore moves runs of them with one copy each.  All or nothing:
 * BSR_E_NOMEM (nothing stored) when fewer than n blocks are free. */
int bsr_store_put_chunks(bsr_ctx* ctx, uint32_t n, const uint64_t* keys, const void* const* group_payloads);

/* Remove the entry (key, group), or all groups of key when group < 0.  Memory
 * in use by a bound request is freed when that request ends.
 * BSR_E_NOTFOUND if no such entry. */
int bsr_store_remove(bsr_ctx* ctx, uint64_t key, int32_t group);

/* Host address, size and stored tag of entry (key, group).  The pointer is
 * valid until the entry is removed or replaced; writing through it models a
 * corrupted external object (the tag is not updated). */
int bsr_store_payload(bsr_ctx* ctx, uint64_t key, uint32_t group, void** host_ptr,
                      uint64_t* nbytes, uint64_t* tag);

/* Number of live (key, group) entries and arena bytes in use. */
int bsr_store_count(bsr_ctx* ctx, uint64_t* n_entries, uint64_t* bytes_used);

/* ---- lower tier: files (§4 "System topology", "Storage-side concurrency is
 * orthogonal"; §6.4 outcome table; §6.5) ---------------------------------------- */

/* Open (create) a file-backed lower tier in directory `dir`: one file per
 * chunk key, a 4 KiB header (magic, key, group mask, per-group tags) then
 * the chunk laid out like a staging slot, padded to 4 KiB.  Files already in
 * the directory with this layout are indexed (the tier outlives processes).
 * Restores read chunk files with load_concurrency reader threads (1..64,
 * the load concurrency of §4) into a pool of readahead_chunks pinned bounce
 * buffers (0 = 2 x load_concurrency; else >= load_concurrency), each reused
 * once the device copy out of it has run.  flags: BSR_FILE_DIRECT. */
int bsr_file_tier_open(bsr_ctx* ctx, const char* dir, uint32_t load_concurrency, uint32_t readahead_chunks,
                       uint32_t flags);

/* Write the chunk of `key` into the file tier (all groups; tags as for
 * bsr_store_put_chunk).  Replaces an existing file. */
int bsr_file_tier_put_chunk(bsr_ctx* ctx, uint64_t key, const void* const* group_payloads);

/* Remove one group's entry (group >= 0) or the whole chunk (group < 0).
 * BSR_E_NOTFOUND if absent. */
int bsr_file_tier_remove(bsr_ctx* ctx, uint64_t key, int32_t group);

/* Number of (key, group) entries in the file tier (0 if not open). */
int bsr_file_tier_count(bsr_ctx* ctx, uint64_t* n_entries);

/* Mark a tier available or not (models a remote store going away).  The
 * probe skips unavailable tiers; a chunk whose tier became unavailable after
 * the probe fails its window as missing. */
int bsr_tier_set_available(bsr_ctx* ctx, int32_t tier, int32_t available);

/* Per-chunk tier chosen by the last probe of `request_id` (BSR_TIER_*; the
 * first available tier holding every group of the chunk), for n_chunks. */
int bsr_plan_tiers(bsr_ctx* ctx, uint64_t request_id, uint8_t* tier_of_chunk, uint32_t n_chunks);

/* ---- the hot path ------------------------------------------------------------- */

/* Probe-only lookup (§3 "Probe globally", §4 probe_only).  Computes the
 * chunk keys of `tokens` (see bsr_chunk_keys) and looks every (key, group)
 * up in the available tiers (the pinned store first, then the file tier).
 * hit_bitmap bit i (LSB-first within byte i/8) is 1 iff one available tier
 * holds every group of chunk i; *n_hit_chunks is the number of leading ones.  Nothing is staged, no reference is kept, and the store is not
 * modified.  If the request carries a force-local marker (§3 "Recover
 * without re-entering the same fault") the result is 0 hits and an all-zero
 * bitmap.  The request's plan (keys, n) is kept for bsr_request_bind.
 * hit_bitmap (ceil(N/8) bytes) and keys_out (N entries) may be NULL. */
int bsr_probe(bsr_ctx* ctx, uint64_t request_id, uint64_t salt, const int32_t* tokens,
              uint64_t n_tokens, uint32_t* n_hit_chunks, uint8_t* hit_bitmap,
              uint64_t* keys_out);

/* Bind a probed request for restore.  Admission: with staging_budget_bytes
 * B = 0 the bind takes the bounded-retrieve lock (BSR_E_BUSY while another
 * request is bound); with B > 0 it is admitted while the rings of the bound
 * requests plus this one (bsr_plan_staging_bytes) stay <= B and a session
 * slot is free (else BSR_E_BUSY, retry after a commit or end; a ring larger
 * than B alone is BSR_E_STAGING).  Concurrently bound requests need their
 * own staging rings and status blocks (overlap -> BSR_E_ARG) and must not
 * share destination blocks; they may share streams.  n_hit_chunks <= the
 * probed n, and n_hit_chunks * chunk_tokens plus twice the largest
 * block_tokens must stay below 2^32 (else BSR_E_ARG).
 * dst: n_groups destinations (block tables are copied to the host once and
 * checked: every id < pool_blocks, no id repeated -> else BSR_E_ARG; with
 * BSR_FLAG_TRUSTED_TABLES they are checked on the device instead, see the
 * flag).
 * staging: device ring of staging_bytes >= bsr_plan_staging_bytes(ctx,
 * n_hit_chunks) (else BSR_E_STAGING); the library uses exactly that many.
 * status: device bsr_dev_status.  Enqueues, on compute_stream, the begin
 * kernel: status reset (fail = 0, q = 1, exposed = 0) and the valid bytes of
 * every advertised block cleared, so no block of the prefix reads valid
 * before commit.  copy_stream and compute_stream must be distinct. */
int bsr_request_bind(bsr_ctx* ctx, uint64_t request_id, uint32_t n_hit_chunks,
                     const bsr_group_dst* dst, void* staging, uint64_t staging_bytes,
                     bsr_dev_status* status, void* copy_stream, void* compute_stream);

/* Restore window [first_chunk, first_chunk + n_chunks) of the bound request
 * (§4 windowed retrieve; 1 <= n_chunks <= W (<= n_hit in whole-plan mode),
 * first_chunk = the next chunk not
 * yet requested).  Asynchronous: for each chunk it looks the entries up
 * (a missing entry, an injected delay beyond the window deadline, or a
 * failed copy submission fails the window), waits for the chunk's slot to be
 * released, and enqueues the pinned-host -> slot copy on copy_stream; per
 * install batch (which may span windows: chunks left over at the end of a
 * call join the next call's batch, and every later call of the request --
 * commit, invalidate, mark, end -- installs them first) it enqueues the
 * install kernel on compute_stream, releases the batch's slots behind it,
 * then enqueues the verify kernel (which reads only the install's tag
 * partials, not the slots).  On a
 * host-detected failure it enqueues the chunks before the failing one, then
 * an invalidate, and returns BSR_E_MISSING / BSR_E_TIMEOUT /
 * BSR_E_TRANSFER; later windows return BSR_E_STATE.  Device-detected
 * corruption is reported by bsr_commit. */
int bsr_restore_window(bsr_ctx* ctx, uint64_t request_id, uint32_t first_chunk,
                       uint32_t n_chunks);

/* The next window of the bound request's plan (§2: the confirmed prefix cut
 * into ordered windows G_1..G_K of at most W chunks, K = ceil(n / W); in
 * whole-plan mode one window of all n): *first_chunk and *n_chunks are what
 * the next bsr_restore_window must pass.  *n_chunks = 0 once every window has
 * been restored, or once the request has failed (nothing more is restored).
 * BSR_E_STATE if the request is not bound. */
int bsr_next_window(bsr_ctx* ctx, uint64_t request_id, uint32_t* first_chunk, uint32_t* n_chunks);

/* Report group `group` of the bound request invalid outside any transfer
 * (its q_g of Eq. 6 becomes 0, e.g. the engine found an erroneous block in
 * that group).  Asynchronous, on compute_stream, after the chunks already
 * restored have been installed and verified (so a corruption among them is
 * still the recorded failure).  From then on every later chunk is past the
 * valid prefix: the device neither installs nor verifies it, and the commit
 * falls back with fail = NONE and q_g = 0 unless an earlier failure was
 * recorded.  Later windows are still accepted; their host-side checks
 * (presence, deadline, transfer) still record the first such failure. */
int bsr_mark_group_invalid(bsr_ctx* ctx, uint64_t request_id, uint32_t group);

/* Request-level commit (Eq. 6 with one rank).  Enqueues the commit kernel:
 * Q = (fail == 0) and q_g for every group.  Q = 1: exposed = n*chunk_tokens
 * and every advertised block's valid byte = 1.  Q = 0: exposed = 0, every
 * advertised block in every group invalid, fallback = 1, and the request's
 * force-local marker is set.  Then waits for the compute stream, reads the
 * status back, releases store references and the request's admission (the
 * lock, or its share of B).
 * Returns BSR_OK in both cases; exposed_tokens / fallback (either may be
 * NULL) report which.  All windows need not have been restored: a commit
 * before the last window exposes nothing (the prefix is incomplete). */
int bsr_commit(bsr_ctx* ctx, uint64_t request_id, uint64_t* exposed_tokens,
               int32_t* fallback);

/* Invalidate the bound request (§3, §4 failed-block and HMA-aware
 * invalidation): enqueues the invalidate kernel (fail = reason if none yet,
 * every advertised block in every group invalid, exposed = 0, fallback = 1)
 * and sets the force-local marker.  Asynchronous and idempotent;
 * bsr_commit or bsr_request_end completes the request.  reason: a
 * BSR_FAIL_* value other than NONE (callers normally pass ABORT). */
int bsr_invalidate(bsr_ctx* ctx, uint64_t request_id, int32_t reason);

/* Successful RUNNING admission of a request: clears its force-local marker. */
int bsr_request_running(bsr_ctx* ctx, uint64_t request_id);

/* Request teardown: completes an uncommitted bound request (waits for its
 * device work), releases references and its admission, clears the
 * force-local marker and forgets the request's plan and counters. */
int bsr_request_end(bsr_ctx* ctx, uint64_t request_id);

/* Counters of the request most recently bound or completed on this context
 * (live while it is bound). */
int bsr_stats_get(bsr_ctx* ctx, bsr_stats* out);

/* Counters of request_id: live while it is bound, then those of its last
 * completion until bsr_request_end or its next probe.  BSR_E_NOTFOUND if
 * the request has neither. */
int bsr_request_stats(bsr_ctx* ctx, uint64_t request_id, bsr_stats* out);

/* Admission state: B, session slots, what is bound now and the peaks. */
int bsr_admission_get(bsr_ctx* ctx, bsr_admission* out);

/* ---- instrumentation ----------------------------------------------------------- */

/* Arm one host-side fault for the next request bound: `kind` BSR_INJECT_*
 * at chunk `chunk` with parameter `param`; BSR_INJECT_NONE disarms. */
int bsr_debug_inject(bsr_ctx* ctx, int32_t kind, uint32_t chunk, uint32_t param);

/* Pinned host -> device bandwidth of this context's device: best of `reps`
 * timed hipMemcpyAsync rounds moving `bytes` from a fresh hipHostMalloc
 * buffer to device memory, split over n_streams streams (1..4).  *gbps in
 * 1e9 B/s.  Needs a GPU context. */
int bsr_measure_h2d(bsr_ctx* ctx, uint64_t bytes, uint32_t n_streams, uint32_t reps,
                    double* gbps);

/* The same link measured with the library's staging-copy kernel: best of
 * `reps` timed launches reading `bytes` (a multiple of 16) from a fresh
 * hipHostMalloc buffer into device memory.  *gbps in 1e9 B/s.  Needs a GPU
 * context. */
int bsr_measure_stage(bsr_ctx* ctx, uint64_t bytes, uint32_t reps, double* gbps);

/* A ceiling for the install kernel: a plain copy of data_bytes / block_bytes
 * whole blocks from a contiguous device buffer into as many distinct blocks
 * of a pool twice the data, drawn in a seeded random order, with the
 * install's workgroup shape, occupancy and XCD work order, and nothing else
 * (no tag, no metadata, no status check).  With BSR_SCATTER_WARM_SOURCE the
 * source is rewritten (a device fill) right before every timed launch, as
 * the staging copy writes a ring slot right before the install reads it;
 * otherwise it is read cold.  Best of `reps` launches; *gbps counts read +
 * write bytes (1e9 B/s).  block_bytes: a positive multiple of 16.  Allocates
 * its own buffers.  Needs a GPU context. */
#define BSR_SCATTER_WARM_SOURCE 1u
int bsr_measure_scatter(bsr_ctx* ctx, uint32_t block_bytes, uint64_t data_bytes, uint32_t reps,
                        uint64_t seed, uint32_t flags, double* gbps);

#ifdef __cplusplus
}
#endif

#endif /* BSR_H */
