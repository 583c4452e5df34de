/*
 * sgdrc.h -- C ABI of the MI355X colour-restricted tensor path.
 *
 * Software-defined resource control in the manner of SGDRC (PPoPP '25):
 * device memory is split into "colours" by an XOR hash of page addresses;
 * tensors are stored on pages of chosen colours through a page-indirection
 * table and read through it by every kernel; each launch runs only on the
 * compute units (CUs) named by a per-stream mask.
 *
 * Conventions for every call below
 * --------------------------------
 *  - Return value: SGDRC_OK (0) or a negative SGDRC_E* code.  On error
 *    nothing is enqueued and no caller memory is touched; the text of the
 *    last error of the calling thread is given by sgdrc_last_error().
 *    Arguments are checked before the context, so argument errors are
 *    reported (SGDRC_EINVAL) even when ctx is NULL.
 *  - Pointers prefixed d_ (and the pool/pt pointers of sgdrc_paged) are
 *    device pointers on the context's device; all others are host pointers.
 *    The caller owns every buffer it passes and keeps it alive until the
 *    enqueued work is done.  The library owns only its context workspace.
 *  - ``stream`` is a hipStream_t handle (NULL = the legacy default stream).
 *    Every operation is asynchronous on that stream except those documented
 *    as waiting: colour_alloc_pagetable and colour_alloc_pagetable_table
 *    (they return the count to the host), sgdrc_suspended,
 *    sgdrc_stream_release, sgdrc_device_error, sgdrc_init and
 *    sgdrc_destroy.
 *  - colour_classify, colour_classify_table, colour_alloc_pagetable_noalloc,
 *    bimodal_relayout, bimodal_relayout_batch, colored_stream and
 *    colored_gemv enqueue kernels only (no memset, copy or host wait), and
 *    every per-launch value travels in the kernel arguments, so they may be
 *    captured into a HIP graph and replayed, except on a stream with an
 *    eviction flag (preemptible launches are resumed from the host).
 *  - Page tables are arrays of uint32 pool-page indices.  Logical byte b of
 *    a paged tensor lives at pool + pt[b >> page_shift] * 2^page_shift +
 *    (b & (2^page_shift - 1)).  Kernels check every page-table entry
 *    against the pool size they are given; an entry out of range is skipped
 *    (its bytes are neither read nor written) and raises the device error
 *    flag SGDRC_DEVERR_PT_RANGE, reported by sgdrc_device_error().
 *  - A context serves one device.  It may be used from several host
 *    threads; operations on one stream are ordered, operations on different
 *    streams may run concurrently (each stream gets its own work queue).
 *  - CU masks (set_cu_mask) confine every tile of work to the allowed CUs.
 *    A launch's remainder below the 16-byte access granularity (the last
 *    n mod 16 bytes of a relayout or triad, the last n mod 16 addresses of
 *    a classify) and, on the ticket queues, any tiles left if no workgroup
 *    reached an allowed CU are handled by the grid's last workgroup, which
 *    may sit on any CU; under the static schedule (see set_cu_mask) a
 *    classify's remainder and histogram total are produced by a
 *    one-workgroup kernel enqueued right after the grid, also on any CU.
 */
#ifndef SGDRC_H
#define SGDRC_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define SGDRC_OK 0
#define SGDRC_EINVAL (-22) /* bad argument */
#define SGDRC_ENOMEM (-12) /* pool holds fewer qualifying pages than requested */
#define SGDRC_ENODEV (-19) /* no usable gfx950 device, or ctx is NULL/not initialised */
#define SGDRC_EHIP (-5)    /* HIP runtime error */

#define SGDRC_MAX_MASKS 8
#define SGDRC_MAX_CUS 256
#define SGDRC_MIN_PAGE_SHIFT 10 /* 1 KiB: the paper's finest colouring granularity (section 6) */
#define SGDRC_MAX_PAGE_SHIFT 30 /* 1 GiB */
#define SGDRC_MAX_BATCH 8

/* device error flags (bitwise OR, sticky until read) */
#define SGDRC_DEVERR_PT_RANGE 1u
#define SGDRC_DEVFLAG_GATE_FALLBACK 2u     /* no workgroup reached an allowed CU; the last did the tiles */
#define SGDRC_DEVERR_SUSPENDED_DROPPED 4u  /* a suspended launch was discarded unresumed */
#define SGDRC_DEVERR_HANDBACK 8u           /* a handed-back tile index out of range (skipped;
                                            * a library fault, never expected) */

/* element encodings */
enum { SGDRC_F32 = 0, SGDRC_BF16 = 1, SGDRC_F16 = 2 };

typedef struct sgdrc_ctx sgdrc_ctx;

/* K XOR masks, 1 <= n_masks <= 8.  Colour bit k of an address a is the
 * parity of (a & masks[k]); bit 0 is the least significant colour bit, so
 * there are 2^K colours.  Masks may only select address bits 0..47. */
typedef struct {
    uint32_t n_masks;
    uint32_t reserved; /* must be 0 */
    uint64_t masks[SGDRC_MAX_MASKS];
} sgdrc_hash;

/* A set of colours: bit c of the 256-bit field (word c/64, bit c%64). */
typedef struct {
    uint64_t bits[4];
} sgdrc_colour_set;

/* A set of logical CUs: bit i = logical CU i, 0 <= i < sgdrc_num_cus().
 * Logical CUs are numbered in (XCC, shader engine, shader array, CU) order,
 * so CUs 32x..32x+31 are the CUs of XCC x on a 256-CU MI355X. */
typedef struct {
    uint64_t bits[4];
} sgdrc_cu_mask;

/* A paged tensor: device pool base (256-byte aligned), device page table,
 * and the pool's capacity in pages (every pt entry must be below it). */
typedef struct {
    void *pool;
    const uint32_t *pt;
    uint64_t pool_pages;
} sgdrc_paged;

/* ---------------------------------------------------------------- context */

/* Create a context on HIP device ``device`` (must be gfx950).  Probes the
 * CU topology by running a kernel that records the XCC_ID and HW_ID
 * registers of every CU, and allocates the context workspace (CU lookup
 * table, per-stream work-queue counters, device error word).  Synchronous. */
int sgdrc_init(int device, sgdrc_ctx **out);

/* Wait for the device, then free the context and its workspace. */
int sgdrc_destroy(sgdrc_ctx *ctx);

/* Number of CUs found by the probe (a negative code if ctx is invalid). */
int sgdrc_num_cus(const sgdrc_ctx *ctx);

/* Hardware identity of logical CU ``cu``: (XCC_ID << 8) | HW_ID[15:8]
 * (the CU, shader-array and shader-engine fields). */
int sgdrc_cu_key(const sgdrc_ctx *ctx, uint32_t cu, uint32_t *key);

/* Text of the calling thread's last error ("" if none). */
const char *sgdrc_last_error(void);

/* Wait for the device, then return and clear the device error flags. */
int sgdrc_device_error(sgdrc_ctx *ctx, uint32_t *flags);

/* Optional per-launch work log, for tests of the CU gate and tile queue.
 * When set, every tile that a kernel processes adds 1 to
 * d_cu_tiles[logical CU] (num_cus entries) and to d_tile_visits[tile index]
 * (tiles beyond tile_cap are not logged).  NULL pointers switch it off.
 * Applies to launches enqueued after the call. */
int sgdrc_set_worklog(sgdrc_ctx *ctx, uint32_t *d_cu_tiles, uint32_t *d_tile_visits,
                      uint64_t tile_cap);

/* Tile count of the last launch enqueued on ``stream`` through this
 * context (0 if none); lets a caller size and read the work log. */
int sgdrc_last_tiles(sgdrc_ctx *ctx, void *stream, uint64_t *tiles);

/* How the last launch enqueued on ``stream`` distributed its tiles:
 * SGDRC_SCHED_QUEUE (atomic ticket queues per group of CUs, with stealing)
 * or SGDRC_SCHED_STATIC (colored_gemv, colour_classify and
 * colour_classify_table under a mask made of whole XCDs: each workgroup
 * derives its tiles from its XCD and index, no atomics).  For tests and
 * tools. */
enum { SGDRC_SCHED_QUEUE = 0, SGDRC_SCHED_STATIC = 1 };
int sgdrc_last_schedule(sgdrc_ctx *ctx, void *stream, uint32_t *schedule);

/* Optional per-launch device time log, for measuring kernel latency without
 * host launch overhead.  Launch i on ``stream`` (counted from this call) of
 * colour_classify, bimodal_relayout, colored_stream or colored_gemv writes
 * two uint64 ticks of the device wall clock to d_slots[2*(i % n_slots)]:
 * the time workgroup 0 (the first one dispatched) started and the time the
 * last workgroup finished.  (Under the static schedule every workgroup
 * records its end in one of 64 partial stamps and a one-wavefront kernel
 * enqueued after the grid writes their maximum.)  d_slots: device memory, 2 * n_slots entries,
 * 8-byte aligned, owned by the caller.  d_slots == NULL switches the log
 * off.  Host-only.  EINVAL: n_slots == 0 with d_slots != NULL, misaligned
 * slots. */
int sgdrc_set_timelog(sgdrc_ctx *ctx, void *stream, uint64_t *d_slots, uint32_t n_slots);

/* Rate of the device wall clock used by the time log, in kHz. */
int sgdrc_wallclock_khz(const sgdrc_ctx *ctx, uint32_t *khz);

/* ------------------------------------------------------------- operations */

/* Cap on the workgroups that later launches on ``stream`` place on each CU
 * (0 = as many as fit, the default).  The hardware sends workgroup i of a
 * grid to XCD i mod (number of XCDs), whatever the CU mask, and a workgroup
 * outside the mask only leaves after it has been placed.  A long persistent
 * kernel that fills its CUs completely would therefore hold back the stray
 * workgroups of short kernels on other streams until it ends; co-located
 * streams give the long-running one a cap below its occupancy to leave room.
 * Host-only.  EINVAL: cap above 64. */
int sgdrc_set_stream_occupancy(sgdrc_ctx *ctx, void *stream, uint32_t max_wgs_per_cu);

/* Tidal compute-unit masking (paper section 7.1, Elastic SM Scaling; the
 * per-launch TPC mask there is replaced by an in-kernel gate).  Sets the CU
 * set used by every later launch on ``stream``: each workgroup reads its
 * CU identity from the hardware registers and exits unless that CU is in
 * the set; the remaining workgroups take tiles from an atomic queue until it
 * is empty.  A colored_gemv or colour_classify under a mask made of whole
 * XCDs (the usual case: all CUs, or n x 32 CUs) needs no queue: the
 * hardware hands
 * workgroup i of a grid to the XCD of workgroup i mod (XCD count), which
 * sgdrc_init checks, so a workgroup on an allowed XCD derives its tiles from
 * its XCD and index alone (SGDRC_SCHED_STATIC).  mask == NULL restores all CUs.  Host-only, takes effect at the
 * next launch, never recreates the stream.  EINVAL: empty mask or a bit at
 * or above sgdrc_num_cus(). */
int set_cu_mask(sgdrc_ctx *ctx, void *stream, const sgdrc_cu_mask *mask);

/* Preemptible best-effort launches (paper section 7.1: a latency-sensitive
 * task preempts the compute units of a best-effort kernel by writing an
 * eviction flag that the persistent kernel polls; the kernel then restarts
 * on fewer units).  With a flag set, later colored_stream and
 * bimodal_relayout launches on ``stream`` are preemptible: each workgroup
 * reads *d_flag at the start of every tile and after claiming the next one
 * and, once it reads non-zero, finishes the tile it is on, hands back a
 * tile it has claimed but not begun, and leaves.  If tiles remain
 * (unclaimed or handed back), the launch ends "suspended": the rest of the
 * work, including the last n mod 16 bytes, waits for sgdrc_resume, whose
 * workgroups take the handed-back tiles first.  Every tile is processed exactly once
 * over a launch and its resumptions, so the result equals an uninterrupted
 * launch.  d_flag: device memory, 4-byte aligned, owned by the caller, who
 * writes it (from the host or from a kernel on another stream) and keeps it
 * alive while such launches may run; a launch started with the flag set
 * does no work.  Preemptible launches use a second work queue of their
 * own; a fresh preemptible launch on a stream whose last one is still
 * suspended first discards that one (and raises SGDRC_DEVERR_SUSPENDED_DROPPED).
 * d_flag == NULL makes later launches non-preemptible (a suspended launch
 * can still be resumed).  Host-only.  EINVAL: misaligned flag, or no work
 * queue left (64 per context, shared with the streams). */
int sgdrc_set_eviction_flag(sgdrc_ctx *ctx, void *stream, const uint32_t *d_flag);

/* Testing aid for preemptible launches: later preemptible launches on
 * ``stream`` and their resumptions behave as if the eviction flag were read
 * as raised at the start of, and after the claim of, any tile whose index
 * is ``tile`` or more (one integer compare per tile, no waiting): the
 * workgroup that starts such a tile finishes it and leaves, and one that
 * has just claimed such a tile hands it back.  This gives tests a mid-run
 * eviction at a chosen point, independent of timing.  tile == 0 switches
 * it off (the default).  Host-only. */
int sgdrc_set_eviction_hook(sgdrc_ctx *ctx, void *stream, uint32_t tile);

/* Forgets everything the context keeps for ``stream`` -- CU mask,
 * workgroup cap, time log, eviction flag and hook, the record of its last
 * preemptible launch -- and returns its work queues to the context, after
 * waiting for the stream.  A suspended launch of the stream that was never
 * resumed is discarded (raising SGDRC_DEVERR_SUSPENDED_DROPPED).  A later
 * use of the same handle starts afresh with all CUs allowed.  Call it
 * before a stream is destroyed or its handle may be handed out again (a
 * stream pool such as PyTorch's reuses handles); a context holds at most
 * 64 work queues at once.  No-op for a stream never used. */
int sgdrc_stream_release(sgdrc_ctx *ctx, void *stream);

/* Enqueues on ``stream`` the continuation of the stream's last preemptible
 * launch, under the stream's current CU mask and eviction flag, with the
 * same arguments (the caller keeps their buffers alive).  If that launch
 * (with its earlier resumptions) has completed, the enqueued kernel does
 * nothing; a resumption can itself be evicted and resumed again.
 * Asynchronous.  EINVAL: no preemptible launch on the stream, or the mask
 * allows no CU. */
int sgdrc_resume(sgdrc_ctx *ctx, void *stream);

/* Enqueues on ``stream`` a one-thread kernel that stores ``value`` to
 * *d_flag (a device-scope store, seen by kernels running on other streams)
 * and, if d_stamp is not NULL, writes the device wall-clock tick of the
 * store to *d_stamp (the clock of sgdrc_set_timelog).  This is how a
 * latency-sensitive stream evicts a best-effort one in stream order (value
 * 1 before its own kernels), and how the best-effort stream clears the
 * flag before resuming (value 0).  EINVAL: d_flag NULL or misaligned,
 * d_stamp misaligned. */
int sgdrc_signal_flag(sgdrc_ctx *ctx, void *stream, uint32_t *d_flag, uint32_t value,
                      uint64_t *d_stamp);

/* Waits for ``stream``, then sets *tiles_left to the number of tiles that
 * the stream's last preemptible launch still has to process: 0 when it has
 * completed, otherwise it is suspended.  EINVAL: no preemptible launch on
 * the stream, NULL tiles_left. */
int sgdrc_suspended(sgdrc_ctx *ctx, void *stream, uint64_t *tiles_left);

/* Sliding-window CU reservation (paper section 7.1): the CUs reserved for
 * the latency-sensitive side are the most that any of the next ``window``
 * queued latency-sensitive kernels needs (ls_cus[i] = CUs that kernel i,
 * in queue order, needs for its best latency; found offline), rounded up
 * to a multiple of ``granule`` CUs (32 = whole XCDs, each with its own L2)
 * and capped at num_cus.  *ls_mask receives the first R logical CUs and
 * *be_mask the others (empty when R = num_cus: the best-effort side is
 * then to be evicted, not masked).  n_queued == 0 gives R = 0.  Pure host
 * computation, no context.  EINVAL: num_cus outside 1..256, window or
 * granule 0, an ls_cus entry above num_cus, NULL pointers. */
int sgdrc_tidal_masks(uint32_t num_cus, const uint32_t *ls_cus, uint32_t n_queued,
                      uint32_t window, uint32_t granule, sgdrc_cu_mask *ls_mask,
                      sgdrc_cu_mask *be_mask);

/* Batched colouring (paper section 6, SPT step 1, marking each page's
 * colour; the hash is the linear XOR form discussed in section 3.2).
 * d_colours[i] = colour(d_addrs[i]) for i < n.  If d_hist != NULL it
 * receives the number of addresses of each colour (2^K uint64 entries,
 * overwritten).  d_addrs and d_colours must be 16-byte aligned, d_hist
 * 8-byte aligned.  n == 0 is valid (hist is zeroed).  EINVAL: bad hash,
 * NULL pointers with n > 0, misaligned pointers. */
int colour_classify(sgdrc_ctx *ctx, const sgdrc_hash *hash, const uint64_t *d_addrs,
                    uint64_t n, uint8_t *d_colours, uint64_t *d_hist, void *stream);

/* Page-table build (paper section 6, SPT steps 2-3, per-colour page lists
 * of a reserved pool).  Pool page i (0 <= i < pool_pages) covers the bytes
 * [a, a + 2^page_shift), a = addr_origin + i * 2^page_shift, and qualifies
 * when every one of those bytes has a colour in ``set`` (section 6 colours
 * whole sectors).  With no mask bit below page_shift that is the colour of
 * a; a mask bit inside the page gives the page's bytes several colours,
 * all of which must be in the set.  Writes to d_pt the first min(found, n_needed) qualifying page
 * indices in ascending order, and sets *n_found = found, the number of
 * qualifying pages in the whole pool.  Returns SGDRC_ENOMEM when
 * found < n_needed (d_pt then holds all ``found`` pages).  Synchronous:
 * returns after the result is in d_pt.  EINVAL: bad hash, page_shift
 * outside [10, 30], addr_origin not page aligned, pool beyond 2^48 bytes of
 * address space, pool_pages > 2^32, n_needed > pool_pages, empty set or
 * a colour >= 2^K in it. */
int colour_alloc_pagetable(sgdrc_ctx *ctx, const sgdrc_hash *hash, uint64_t addr_origin,
                           uint32_t page_shift, uint64_t pool_pages,
                           const sgdrc_colour_set *set, uint64_t n_needed, uint32_t *d_pt,
                           uint64_t *n_found, void *stream);

/* colour_alloc_pagetable for callers that cannot allocate: code under HIP
 * graph capture, tight serving loops, harnesses that forbid hipMalloc.  It
 * allocates nothing and never waits for the device: the same table as
 * colour_alloc_pagetable goes to d_pt, but the call is asynchronous on
 * ``stream``, the count of qualifying pages in the pool goes to *d_n_found
 * (device memory, one uint64, 8-byte aligned) instead of a host variable,
 * and a shortfall is no error: the caller compares *d_n_found with
 * n_needed (d_pt then holds all the qualifying pages).  Its scratch is a
 * fixed 192.25 KiB block of the library's own device memory, one per
 * device and held until the process ends, which limits pool_pages to 2^26.
 * Every call on a device shares that block: calls that overlap on one GPU
 * (on different streams or host threads) race, and the caller must order
 * them.  Every scratch word a call reads is first written by the same
 * call, so nothing needs clearing between calls.  EINVAL: as
 * colour_alloc_pagetable, pool_pages above 2^26, d_n_found NULL or
 * misaligned. */
int colour_alloc_pagetable_noalloc(sgdrc_ctx *ctx, const sgdrc_hash *hash, uint64_t addr_origin,
                                   uint32_t page_shift, uint64_t pool_pages,
                                   const sgdrc_colour_set *set, uint64_t n_needed, uint32_t *d_pt,
                                   uint64_t *d_n_found, void *stream);

/* A colour table (paper section 5.3: for hashes that are not XOR-linear, a
 * table made offline holds the channel of every 1 KiB partition): lut[i]
 * (device memory) is the colour of the bytes [origin + i 2^shift,
 * origin + (i + 1) 2^shift); 255 means no colour, as does any address
 * outside the table. */
typedef struct {
    const uint8_t *lut;
    uint64_t origin;
    uint64_t entries;
    uint32_t shift;     /* log2 of the partition size, 8..30 */
    uint32_t reserved;  /* must be 0 */
} sgdrc_colour_table;

/* colour_classify through a colour table: d_colours[i] = the colour of
 * d_addrs[i] (255 if none); d_hist (nullable, 256 entries) counts every
 * colour value, 255 included.  Same launch, gate and alignment rules as
 * colour_classify.  EINVAL: NULL table, shift outside 8..30, reserved not
 * 0, entries without a table pointer, a table past 2^48, NULL or
 * misaligned buffers. */
int colour_classify_table(sgdrc_ctx *ctx, const sgdrc_colour_table *table,
                          const uint64_t *d_addrs, uint64_t n, uint8_t *d_colours,
                          uint64_t *d_hist, void *stream);

/* colour_alloc_pagetable through a colour table: pool page i, the bytes
 * [a, a + 2^page_shift) with a = addr_origin + i 2^page_shift, qualifies
 * when every partition it touches lies in the table and has a colour in the
 * set.  Pages smaller than a partition (page_shift < shift) take the
 * colour of their partition.  Synchronous, ENOMEM on shortfall, as
 * colour_alloc_pagetable; EINVAL as there (the set may not name colour
 * 255) and as colour_classify_table for the table. */
int colour_alloc_pagetable_table(sgdrc_ctx *ctx, const sgdrc_colour_table *table,
                                 uint64_t addr_origin, uint32_t page_shift, uint64_t pool_pages,
                                 const sgdrc_colour_set *set, uint64_t n_needed, uint32_t *d_pt,
                                 uint64_t *n_found, void *stream);

/* Bimodal relayout (paper section 7.2, moving a tensor between its
 * all-channel and its restricted page set): copies n_bytes logical bytes,
 * logical byte b going from src's page pt[b >> s] to dst's page
 * pt[b >> s] at the same in-page offset.  Both tables hold
 * ceil(n_bytes / 2^page_shift) entries.  Bytes of dst pages beyond n_bytes
 * are not written.  src and dst must not overlap.  EINVAL: NULL pointers,
 * pools not 256-byte aligned, page_shift outside [10, 30]. */
int bimodal_relayout(sgdrc_ctx *ctx, const sgdrc_paged *dst, const sgdrc_paged *src,
                     uint64_t n_bytes, uint32_t page_shift, void *stream);

/* One copy of a batched relayout. */
typedef struct {
    sgdrc_paged dst;
    sgdrc_paged src;
    uint64_t n_bytes;
    uint32_t page_shift;
    uint32_t reserved; /* 0 */
} sgdrc_relayout_item;

/* Batched bimodal relayout (paper section 7.2: on a change of co-location
 * state every latency-sensitive tensor moves): the n_items copies of
 * ``items``, each exactly as bimodal_relayout would make it, in one launch
 * per 32 items instead of one per tensor.  Items may differ in page size;
 * no item's destination may overlap another item's source or destination.
 * Always a plain launch (not preemptible, even on a stream with an
 * eviction flag).  n_items == 0 launches nothing.  Asynchronous; ``items`` is
 * read before the call returns.  EINVAL: items NULL with n_items > 0, an
 * item invalid as for bimodal_relayout, reserved not 0, more than 2^31
 * 64 KiB tiles in one launch. */
int bimodal_relayout_batch(sgdrc_ctx *ctx, const sgdrc_relayout_item *items, uint32_t n_items,
                           void *stream);

/* Colour-restricted streaming triad (paper section 6, SPT step 4, the
 * re-indexed vector kernel): a[i] = fmaf(s, c[i], b[i]) for i < n_elems,
 * one rounding, every fp32 element reached through its array's page table
 * (ceil(4 n_elems / 2^page_shift) entries each).  a may alias b or c
 * element-for-element (same pool and table) but must not otherwise overlap
 * them.  EINVAL: as for bimodal_relayout. */
int colored_stream(sgdrc_ctx *ctx, const sgdrc_paged *a, const sgdrc_paged *b,
                   const sgdrc_paged *c, float s, uint64_t n_elems, uint32_t page_shift,
                   void *stream);

/* Colour-restricted GEMV / small-batch GEMM of a memory-bound layer (paper
 * section 7.2): d_y[b*M + m] = sum_k W[m][k] * x[b][k], fp32 result,
 * products summed in fp32.  W is row-major [M x K] of w_dtype, stored
 * through w's page table (ceil(M K esize / 2^page_shift) entries); d_x is
 * contiguous [batch x K] of x_dtype (16-byte aligned); d_y is contiguous
 * [batch x M] fp32.  Batches 3..8 with bf16 x bf16 or f16 x f16 operands
 * run on MFMA; all other cases on the vector ALUs.  The sum order depends
 * only on (M, K, batch, dtypes), never on the CU mask, so results are
 * bitwise reproducible.  EINVAL: batch outside 1..8, M or K zero, K *
 * esize(w_dtype) not a multiple of 16, x of 4 GiB or more, a tile's rows
 * (4, or 16 on MFMA) spanning more pages than one tile stages (256), unknown
 * dtype, NULL pointers, unaligned pointers. */
int colored_gemv(sgdrc_ctx *ctx, const sgdrc_paged *w, int w_dtype, uint32_t M, uint32_t K,
                 const void *d_x, int x_dtype, uint32_t batch, float *d_y,
                 uint32_t page_shift, void *stream);

/* The launch plan colored_gemv uses for a shape, given the number of CUs
 * the stream's mask allows (host-only, no context, no device): the kernel
 * path (vector ALUs or MFMA), rows of W per tile, loads in flight (vector
 * path: 16-byte loads per lane and row; MFMA: register sets of 2 KiB row
 * chunks), the batch columns the kernel is compiled for, the tile count,
 * x_once (1 when each workgroup loads x once: on the vector path into
 * registers, for rows that one round of loads covers; on the MFMA path the
 * whole K into LDS, at batch 3-4 with rows of at most 8 KiB; it changes no
 * result), and sum_depth: the most roundings any product W[m][k] x[b][k]
 * meets on its way into y (the fp32 additions and FMAs of the kernel's fixed summation
 * tree, each MFMA counted as up to 32 additions), so that
 * |y - exact| <= sum_depth * 2^-24 * sum_k |W[m][k] x[b][k]| to first order
 * (products of bf16 or f16 operands are exact in fp32).  Lets tests and
 * tools see which kernel a configuration runs.  EINVAL: allowed_cus outside
 * 1..256, NULL out, or a shape colored_gemv rejects. */
enum { SGDRC_GEMV_VALU = 0, SGDRC_GEMV_MFMA = 1 };
typedef struct {
    uint32_t path;
    uint32_t rows;
    uint32_t loads;
    uint32_t batch_cols;
    uint64_t tiles;
    uint32_t sum_depth;
    uint32_t x_once;
} sgdrc_gemv_plan;

int colored_gemv_plan(uint32_t allowed_cus, int w_dtype, uint32_t M, uint32_t K, int x_dtype,
                    uint32_t batch, sgdrc_gemv_plan *out);

/* ---------------------------------------------------- bimodal tensors
 *
 * Host runtime for the paper's bimodal tensors (section 7.2): which page
 * set every tensor argument of a kernel uses, by tensor class and by the
 * co-location state, and the moves between page sets when the state
 * changes.  Each tensor has two forms given by the caller: ``all_form``
 * (a page set over all channels, e.g. an identity table over a plain
 * buffer) and ``part_form`` (a coloured page set: the best-effort colours
 * for best-effort tensors, the latency-sensitive colours for
 * latency-sensitive ones), both able to hold n_bytes.
 *
 *  SGDRC_BM_BE_WEIGHT   memory-bound best-effort input: two resident copies
 *                       (registration fills part_form from all_form); read
 *                       from all_form in SGDRC_BM_MONOPOLY, from part_form
 *                       in SGDRC_BM_COLOCATED; never written.
 *  SGDRC_BM_LS_TENSOR   memory-bound latency-sensitive tensor: one copy,
 *                       given in all_form at registration, kept in
 *                       part_form while COLOCATED and in all_form while
 *                       MONOPOLY (sgdrc_bm_set_state moves it).
 *  SGDRC_BM_ACTIVATION  intermediate result buffer (capacity n_bytes):
 *                       written in the form of the writing kernel's state
 *                       and read from where it was last written; reused
 *                       through sgdrc_bm_acquire / sgdrc_bm_release.
 *
 * Moves are relayout launches on the given stream (a state change moves
 * every latency-sensitive tensor with one bimodal_relayout_batch); the caller
 * orders them against the kernels that use the tensors and keeps all
 * buffers alive.  Thread-safe.  Errors as elsewhere; a NULL or destroyed
 * runtime gives EINVAL. */
typedef struct sgdrc_bimodal sgdrc_bimodal;
enum { SGDRC_BM_BE_WEIGHT = 0, SGDRC_BM_LS_TENSOR = 1, SGDRC_BM_ACTIVATION = 2 };
enum { SGDRC_BM_MONOPOLY = 0, SGDRC_BM_COLOCATED = 1 };  /* states */
enum { SGDRC_BM_ALL = 0, SGDRC_BM_PART = 1 };            /* forms */

/* New runtime in state SGDRC_BM_MONOPOLY.  ctx may be NULL: such a runtime
 * holds activations only (no moves).  Host-only. */
int sgdrc_bm_create(sgdrc_ctx *ctx, sgdrc_bimodal **out);
int sgdrc_bm_destroy(sgdrc_bimodal *bm);

/* Registers a tensor of class ``cls`` (see above); *id receives its index
 * (0, 1, ... in registration order).  A BE weight's part_form copy, and an
 * LS tensor's move when the runtime is COLOCATED, are enqueued on
 * ``stream``.  EINVAL: unknown class, bad forms or page_shift, n_bytes 0,
 * NULL id; ENODEV: a weight or LS tensor on a runtime without context. */
int sgdrc_bm_register(sgdrc_bimodal *bm, uint32_t cls, const sgdrc_paged *all_form,
                      const sgdrc_paged *part_form, uint64_t n_bytes, uint32_t page_shift,
                      void *stream, uint32_t *id);

/* Changes the state; on a change every LS tensor moves to its form for the
 * new state (relayouts on ``stream``).  EINVAL: unknown state. */
int sgdrc_bm_set_state(sgdrc_bimodal *bm, int state, void *stream);
int sgdrc_bm_state(sgdrc_bimodal *bm, int *state);

/* The descriptor a kernel reads tensor ``id`` through, and (if ``where``
 * is not NULL) which form it is.  EINVAL: unknown id, or an activation not
 * written since it was acquired. */
int sgdrc_bm_input(sgdrc_bimodal *bm, uint32_t id, sgdrc_paged *out, int *where);

/* The descriptor a kernel writes tensor ``id`` through: for an activation
 * the form of the current state, recorded as where it now lives; for an
 * LS tensor its current form.  EINVAL: unknown id, a BE weight. */
int sgdrc_bm_output(sgdrc_bimodal *bm, uint32_t id, sgdrc_paged *out, int *where);

/* Takes the free activation with the smallest capacity of at least
 * n_bytes (lowest id among equals); its contents count as unwritten.
 * ENOMEM: none free.  Release returns it to the free list (EINVAL if it is
 * not an acquired activation). */
int sgdrc_bm_acquire(sgdrc_bimodal *bm, uint64_t n_bytes, uint32_t *id);
int sgdrc_bm_release(sgdrc_bimodal *bm, uint32_t id);

#ifdef __cplusplus
}
#endif

#endif /* SGDRC_H */
