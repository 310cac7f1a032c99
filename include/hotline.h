/*
 * hotline.h -- C ABI of libhotline.so, the MI355X (gfx950) hot path of the
 * Hotline heterogeneous recommendation-training pipeline ("Heterogeneous
 * Acceleration Pipeline for Recommendation System Training", arXiv 2204.05436).
 *
 * Conventions (all entry points):
 *  - Pointers are DEVICE pointers unless marked (host).  w_host is a pointer
 *    the GPU can dereference to the pinned, device-mapped host table
 *    (hl_host_alloc returns one).
 *  - The caller owns every buffer, including workspaces; the handle owns only
 *    its profiling and hot-set state.  No call allocates memory after
 *    hl_create (hl_host_alloc / hl_workspace_* aside).
 *  - Calls are asynchronous and stream-ordered on `stream` (a hipStream_t;
 *    NULL = the null stream) unless stated otherwise.  A handle and a
 *    workspace are not thread-safe and belong to one stream at a time.
 *  - Argument errors found on the host return synchronously (HL_ERR_*) and
 *    enqueue nothing.  Errors found by a kernel (an id outside the tables, a
 *    code naming no row, staging overflow) set bits of the handle's device
 *    error word (HL_DEVERR_*), read with hl_last_device_error; outputs of the
 *    call are then unspecified, except where stated.
 *  - Lookup layout (sample-major CSR): bag index = (b*steps + s)*n_tables + t;
 *    sample b owns bags [b*bps, (b+1)*bps) where bps = bags_per_sample;
 *    bag_ptr[n_bags+1] (int32) indexes the per-lookup arrays; the table of
 *    bag j is j % n_tables.
 *  - Row ids: gid = (rows of tables before t) + row, < 2^32-1.
 *  - Slot codes (int32): [0, n_hot) = hot-cache slot (the row's rank among
 *    the ascending hot ids); [k_cap, k_cap + staging rows) = staging row of a
 *    gathered cold row; -1 = cold row not yet gathered (invalid for the
 *    embedding calls).
 *  - Embedding rows: dim elements of fp32 or bf16 (storage); pooled outputs
 *    and gradients are always fp32, [n_bags, dim] row-major.
 */
#ifndef HOTLINE_H
#define HOTLINE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  HL_OK = 0,
  HL_ERR_INVALID_ARG = 1,  /* bad pointer/size/shape found on the host */
  HL_ERR_OUT_OF_RANGE = 2, /* a value outside its table or capacity (host-checked) */
  HL_ERR_CAPACITY = 3,     /* a buffer or workspace is too small */
  HL_ERR_HIP = 4,          /* the HIP runtime reported an error */
  HL_ERR_UNSUPPORTED = 5,  /* shape or dtype the library does not handle */
  HL_ERR_DEVICE = 6        /* hl_last_device_error: the device error word is set */
} hl_status;

/* bits of the device error word */
#define HL_DEVERR_OUT_OF_RANGE 0x1u /* a table row >= its table's rows, or a gid >= n_rows */
#define HL_DEVERR_BAD_CODE 0x2u     /* a slot code naming no row in an embedding call */
#define HL_DEVERR_CAPACITY 0x4u     /* cold rows exceed the staging capacity */
#define HL_DEVERR_BAD_HOTSET 0x8u   /* hl_set_hot: ids not strictly ascending or >= n_rows */
#define HL_DEVERR_STALL 0x10u       /* a cross-block wait hit its spin limit (never expected) */
#define HL_DEVERR_SHAPE 0x20u       /* bag_ptr[n_bags] differs from the n_lookups passed */
#define HL_DEVERR_INTERNAL 0x40u    /* an internal bound check failed (never expected); the write was skipped */

typedef enum { HL_F32 = 0, HL_BF16 = 1 } hl_dtype;

typedef struct hl_handle hl_handle;
typedef void* hl_stream; /* hipStream_t */

/* A static string naming status s; any int32 value is accepted (an unknown
 * one gives "unknown status"). */
const char* hl_status_string(int32_t s);

/* ---------------------------------------------------------------- handle --
 * Tables and their base registers: the accelerator's Address Registers hold
 * each table's base (Sec. V-A "Data Dispatcher"; s_wr of the ISA table).
 * rows_per_table (host, n_tables entries) fixes gid = base[t] + row; total
 * rows must be < 2^32-1.  k_cap is the hot-cache capacity in rows (>= 1).
 * dtype is one of hl_dtype's values, passed as a plain int32 so that any value
 * a caller hands over is defined: any other value gives HL_ERR_INVALID_ARG.
 * Allocates the handle's device state on the current device: access counts
 * (4 B/row), hot-set bitmap (1 bit/row) and rank directory (4 B per 256 rows).
 * Synchronous. */
hl_status hl_create(hl_handle** out, int32_t n_tables, const uint32_t* rows_per_table, int32_t dim,
                    int32_t dtype, uint32_t k_cap);
hl_status hl_destroy(hl_handle* h);
uint64_t hl_n_rows(const hl_handle* h);
uint32_t hl_n_hot(const hl_handle* h);   /* size of the current hot set (host copy) */
uint32_t hl_k_cap(const hl_handle* h);

/* Workspace bytes for calls with up to max_lookups lookups, max_bags bags and
 * max_samples samples.  A workspace must be zero-filled once before its first
 * use (hl_workspace_init, or any zero fill) and then belongs to this handle;
 * the calls keep it reusable.  Used by hl_partition, hl_cold_plan /
 * hl_cold_gather and hl_embbag_bwd_plan / _apply / _sgd, never two of them
 * concurrently; hl_cold_fetch and hl_cold_scatter do not touch it. */
size_t hl_workspace_bytes(const hl_handle* h, int64_t max_lookups, int64_t max_bags,
                          int32_t max_samples);
hl_status hl_workspace_init(void* workspace, size_t bytes, hl_stream stream);

/* ----------------------------------------------------- address generation --
 * gids[i] = base[table of lookup i] + rows[i] for the n_bags bags of bag_ptr
 * (Sec. V-A: the memory controller forms row addresses from the Address
 * Registers).  A row >= its table's size yields gid 0xFFFFFFFF and sets
 * HL_DEVERR_OUT_OF_RANGE. */
hl_status hl_lookup_gids(const hl_handle* h, const uint32_t* rows, const int32_t* bag_ptr,
                         int64_t n_bags, uint32_t* gids, hl_stream stream);

/* ------------------------------------------------------------- profiling --
 * Learning phase (Sec. IV "The Learning Phase"; Sec. V-B Embedding Access
 * Logger): counts[gid] += 1 for each of the n lookups of a sampled
 * mini-batch, duplicates included.  Ids >= n_rows are skipped and set
 * HL_DEVERR_OUT_OF_RANGE. */
hl_status hl_profile_count(hl_handle* h, const uint32_t* gids, int64_t n, hl_stream stream);

/* Copy the access counts (n_rows uint32) to counts_out. */
hl_status hl_profile_counts(const hl_handle* h, uint32_t* counts_out, hl_stream stream);

/* Hot set = the k most accessed rows (exact counts: the "Oracle LFU" the paper
 * measures its tracker against, Sec. V-B), among rows accessed at least once,
 * ties to the smaller id; n_hot = min(k, #accessed), k <= k_cap.  Writes the
 * hot ids in ascending order to hot_ids_out (device, >= min(k, n_rows)
 * entries), rebuilds the membership bitmap and rank directory, stores n_hot in
 * the handle and in *n_hot_out (host).  reset_counts != 0 zeroes the counts
 * afterwards.  Synchronous (waits for `stream`). */
hl_status hl_profile_topk(hl_handle* h, uint32_t k, uint32_t* hot_ids_out, uint32_t* n_hot_out,
                          int reset_counts, hl_stream stream);

/* Install an explicit hot set: n_hot strictly ascending ids < n_rows (device).
 * Rebuilds bitmap and rank directory; n_hot <= k_cap.  Violations set
 * HL_DEVERR_BAD_HOTSET (the set is then unspecified). */
hl_status hl_set_hot(hl_handle* h, const uint32_t* hot_ids, uint32_t n_hot, hl_stream stream);

/* Fill the hot cache: w_hot[s] = w_host[hot_ids[s]] for s < n_hot (the hot
 * rows are copied to GPU memory after learning, Sec. IV). */
hl_status hl_hot_fill(const hl_handle* h, const uint32_t* hot_ids, const void* w_host, void* w_hot,
                      hl_stream stream);
/* The Embedding Access Logger with SRRIP replacement (Sec. V-B: a cache of
 * row ids with a 2-bit re-reference prediction value per entry, in place of a
 * counter per row; compared with exact counting, the "Oracle LFU", in the
 * paper's tracker figure).  n_sets sets of `ways` ways (1..16); row id g lives
 * in set mix(g) % n_sets, mix being the 32-bit finalizer of MurmurHash3; a hit
 * sets the entry's value to 0; a miss takes the first way whose value is 3,
 * ageing every way of the set by one until one is, and enters with 2; empty
 * ways hold 3.  hl_eal_access feeds one batch of row ids (device, in lookup
 * order; an id 0xFFFFFFFF is skipped) in stream order, asynchronously on
 * `stream`; batches take effect in call order.  hl_eal_hot writes every id the
 * logger holds, ascending, to hot_ids_out (device, n_sets * ways entries) and
 * their number to *n_hot_out (host; synchronous): a hot set for hl_set_hot.
 * hl_eal_state copies the entries (ids, values; set-major, n_sets * ways each,
 * device) for inspection.  hl_eal_create allocates the logger (empty) and its
 * workspace for up to max_lookups ids per call; HL_ERR_CAPACITY: more ids in
 * one call; HL_ERR_INVALID_ARG: ways outside 1..16, n_sets 0, NULL. */
typedef struct hl_eal hl_eal;
hl_status hl_eal_create(hl_handle* h, uint32_t n_sets, int32_t ways, int64_t max_lookups, hl_eal** out);
hl_status hl_eal_destroy(hl_eal* e);
hl_status hl_eal_reset(hl_eal* e, hl_stream stream);
hl_status hl_eal_access(hl_eal* e, const uint32_t* gids, int64_t n, hl_stream stream);
hl_status hl_eal_hot(hl_eal* e, uint32_t* hot_ids_out, uint32_t* n_hot_out, hl_stream stream);
hl_status hl_eal_state(const hl_eal* e, uint32_t* tags_out, uint8_t* rrpv_out, hl_stream stream);

/* Hot-set migration of the recurring learning phase (Sec. V-B: the EAL
 * switches back to learning from time to time; Sec. VI: twice per epoch;
 * Sec. IV: hot rows are trained on the GPU, the others in CPU memory).  Call
 * it after hl_profile_topk (or hl_set_hot) has replaced the hot set
 * old_ids[0..n_old) (device, ascending: the set w_hot_old holds, row s in slot
 * s) by new_ids[0..hl_n_hot(h)) (device, ascending: that call's hot ids).  It
 * fills w_hot_new (device, at least hl_n_hot(h) rows, not overlapping
 * w_hot_old): a row in both sets is copied from its old slot, a row only in
 * the new set is read from w_host; and every row only in the old set is
 * written back to w_host (the pinned host table, device-visible pointer, as in
 * hl_cold_fetch).  The table as the path reads it, a hot row from the cache
 * and any other from w_host, is thus unchanged, bit for bit.  Asynchronous on
 * `stream`; nothing else may use the three tables meanwhile.  HL_ERR_CAPACITY:
 * n_old > k_cap; HL_ERR_INVALID_ARG: NULL where rows are needed, or the caches
 * overlap.  An id >= n_rows sets HL_DEVERR_BAD_HOTSET and its row is skipped. */
hl_status hl_hot_migrate(const hl_handle* h, const uint32_t* old_ids, uint32_t n_old, const uint32_t* new_ids,
                         const void* w_hot_old, void* w_hot_new, void* w_host, hl_stream stream);

/* Mini-batch shape used below: n_samples samples of bags_per_sample bags,
 * bag_ptr[n_samples*bags_per_sample + 1] (device), and n_lookups (host) =
 * bag_ptr[n_samples*bags_per_sample] (a mismatch sets HL_DEVERR_SHAPE).
 * Sample selection (mu-batch calls): sample_ids == NULL selects samples
 * 0..n_sel_max-1 (every sample when n_sel_max = n_samples); otherwise
 * sample_ids[0..n) with n = *n_sel_dev when n_sel_dev is not NULL (a device
 * count, e.g. from hl_partition) else n_sel_max; n must not exceed
 * n_sel_max. */

/* -------------------------------------------------------- classification --
 * flags[b] = 1 iff every lookup of sample b names a hot row, else 0 (a single
 * non-hot lookup makes the input non-popular: Sec. I insight 2, Sec. V-C
 * Lookup Engine).  A sample without lookups is popular. */
hl_status hl_classify(const hl_handle* h, const uint32_t* gids, const int32_t* bag_ptr,
                      int32_t n_samples, int32_t bags_per_sample, int64_t n_lookups, uint8_t* flags,
                      hl_stream stream);

/* Mini-batch fragmentation into the popular and non-popular mu-batches, with
 * O u X = M and O n X = {} (Sec. IV-A, Eq. 3): pop_ids = ascending samples with
 * flag 1, nonpop_ids = ascending samples with flag 0 (each list sized
 * n_samples).  counts_dev[0] = |O|, counts_dev[1] = |X| (device). */
hl_status hl_partition(hl_handle* h, const uint8_t* flags, int32_t n_samples, int32_t* pop_ids,
                       int32_t* nonpop_ids, int32_t* counts_dev, void* workspace, size_t ws_bytes,
                       hl_stream stream);

/* Address generation of the Data Dispatcher (Sec. V-A: each lookup is turned
 * into the address of its row; Sec. IV: the hot rows live in GPU memory, the
 * others in CPU memory): codes[i] = hot-cache slot of gids[i] (the rank of
 * gids[i] among the ascending hot ids), or -1 when the row is not hot (its
 * address is resolved by the cold gather).  gids and codes hold n entries
 * (device); an id >= n_rows gives -1 and sets HL_DEVERR_OUT_OF_RANGE. */
hl_status hl_remap(const hl_handle* h, const uint32_t* gids, int64_t n, int32_t* codes,
                   hl_stream stream);

/* The Data Dispatcher of Sec. V-A in one pass over the mini-batch: the
 * results of hl_lookup_gids (gids), hl_classify (flags), hl_partition
 * (pop_ids, nonpop_ids, counts_dev) and hl_remap (codes), bit for bit, with
 * the same error behaviour.  The workspace (hl_workspace_bytes) holds its
 * cross-block state in the header; mini-batches too large for that state take
 * the four calls in turn. */
hl_status hl_dispatch(hl_handle* h, const uint32_t* rows, const int32_t* bag_ptr, int32_t n_samples,
                      int32_t bags_per_sample, int64_t n_lookups, uint32_t* gids, int32_t* codes,
                      uint8_t* flags, int32_t* pop_ids, int32_t* nonpop_ids, int32_t* counts_dev,
                      void* workspace, size_t ws_bytes, hl_stream stream);

/* ------------------------------------------------------------ cold gather --
 * Working parameters of a mu-batch (Sec. V-A: DMA reads of non-hot rows from
 * CPU memory; dma_rd of the ISA).  Over the lookups of the selected samples
 * whose code is -1: cold_ids_out = their distinct gids in order of first
 * occurrence in the mini-batch's lookup (CSR) order, which for a selection in
 * ascending sample order is the order a stream over the mu-batch meets them;
 * each such code becomes k_cap + (index in cold_ids_out); staging[u] =
 * w_host[cold_ids[u]] bit for bit (rows read by the GPU over the host link).
 * n_cold_dev (device) receives the number of cold rows.  If it exceeds
 * staging_cap_rows the call sets HL_DEVERR_CAPACITY and writes nothing but
 * n_cold_dev and workspace.  Lookups whose code is not -1 are left alone. */
hl_status hl_cold_gather(hl_handle* h, const uint32_t* gids, int32_t* codes, const int32_t* bag_ptr,
                         int32_t n_samples, int32_t bags_per_sample, int64_t n_lookups,
                         const int32_t* sample_ids, const int32_t* n_sel_dev, int32_t n_sel_max,
                         const void* w_host, void* staging, int32_t staging_cap_rows,
                         uint32_t* cold_ids_out, int32_t* n_cold_dev, void* workspace,
                         size_t ws_bytes, hl_stream stream);

/* The two halves of hl_cold_gather, for the paper's pipeline (Sec. IV and the
 * pipeline figure: the working parameters of the non-popular mu-batch are
 * gathered while the popular mu-batch runs).  hl_cold_plan does everything
 * but the row copy: cold_ids_out, n_cold_dev and the code rewrite, with the
 * same capacity rule.  hl_cold_fetch then copies staging[u] =
 * w_host[cold_ids[u]] for u < *n_cold_dev (device count); it reads only its
 * arguments, not the workspace, so once the plan has completed it may run on
 * another stream concurrently with any other call except those that write
 * cold_ids, n_cold_dev or staging.  A count above staging_cap_rows copies
 * nothing and sets HL_DEVERR_CAPACITY; an id >= n_rows is skipped and sets
 * HL_DEVERR_OUT_OF_RANGE. */
hl_status hl_cold_plan(hl_handle* h, const uint32_t* gids, int32_t* codes, const int32_t* bag_ptr,
                       int32_t n_samples, int32_t bags_per_sample, int64_t n_lookups,
                       const int32_t* sample_ids, const int32_t* n_sel_dev, int32_t n_sel_max,
                       int32_t staging_cap_rows, uint32_t* cold_ids_out, int32_t* n_cold_dev,
                       void* workspace, size_t ws_bytes, hl_stream stream);
hl_status hl_cold_fetch(hl_handle* h, const uint32_t* cold_ids, const int32_t* n_cold_dev,
                        int32_t staging_cap_rows, const void* w_host, void* staging, hl_stream stream);

/* Allocates now (and zero-fills on `stream`) the handle's cold-gather hash
 * table for calls of up to max_lookups lookups, which hl_cold_plan would
 * otherwise allocate on first use; callers that capture the plan into a graph
 * reserve first. */
hl_status hl_cold_reserve(hl_handle* h, int64_t max_lookups, hl_stream stream);

/* Write-back of the updated working parameters (Sec. IV: non-hot rows are
 * updated in CPU main memory by DMA; dma_wr of the ISA): w_host[cold_ids[u]] =
 * staging[u] bit for bit, for u < *n_cold_dev, over the host link.  The ids
 * must be distinct (hl_cold_plan's are).  Same count and id rules as
 * hl_cold_fetch; reads no workspace. */
hl_status hl_cold_scatter(hl_handle* h, const uint32_t* cold_ids, const int32_t* n_cold_dev,
                          int32_t staging_cap_rows, const void* staging, void* w_host,
                          hl_stream stream);

/* -------------------------------------------------------------- embedding --
 * Sum pooling (Sec. V-D Reducer, sparse-length element-wise sum; v_add of the
 * ISA): out[bag] = sum over the bag's lookups of row(code) accumulated in fp32
 * (bf16 rows widened exactly), for every bag of the selected samples,
 * written at the bag's own position of out [n_samples*bags_per_sample, dim].  row(c) = w_hot[c] for c < n_hot, staging[c - k_cap]
 * for k_cap <= c < k_cap + staging_rows; any other code sets HL_DEVERR_BAD_CODE
 * and contributes nothing.  An empty bag pools to zero. */
hl_status hl_embbag_fwd(const hl_handle* h, const void* w_hot, const void* staging,
                        int32_t staging_rows, const int32_t* codes, const int32_t* bag_ptr,
                        int32_t n_samples, int32_t bags_per_sample, int64_t n_lookups,
                        const int32_t* sample_ids, const int32_t* n_sel_dev, int32_t n_sel_max,
                        float* out, hl_stream stream);

/* hl_embbag_fwd in halves (the non-popular mu-batch's hot rows are in GPU
 * memory before its working parameters arrive, Sec. IV): a bag's sum takes its
 * hot rows first, then its staging rows, each in lookup order, so that part 1
 * (hot rows only; out = the partial sum, 0 for a bag without hot rows) followed
 * by part 2 (staging rows only, added onto out; bags without staging rows are
 * not touched) gives out bit for bit as part 0 (hl_embbag_fwd) does.  Part 1
 * reads no staging row. */
hl_status hl_embbag_fwd_part(const hl_handle* h, const void* w_hot, const void* staging,
                             int32_t staging_rows, const int32_t* codes, const int32_t* bag_ptr,
                             int32_t n_samples, int32_t bags_per_sample, int64_t n_lookups,
                             const int32_t* sample_ids, const int32_t* n_sel_dev, int32_t n_sel_max,
                             float* out, int32_t part, hl_stream stream);

/* Backward of sum pooling plus one SGD step with duplicate rows coalesced
 * (hot rows updated in GPU memory, Sec. IV): for every distinct code c among
 * the selected bags' lookups, G_c = sum of dY[bag(i)] over its lookups and
 * row(c) <- round_storage(row(c) - lr * G_c), round to nearest even.  Each
 * row is written once; rows no lookup names are untouched.  Deterministic:
 * the summation order depends only on the inputs (ascending lookup order).
 * dY: [n_samples * bags_per_sample, dim] fp32.  Invalid codes set
 * HL_DEVERR_BAD_CODE and are skipped.  A mini-batch with as many lookups as
 * bags is taken to hold one lookup per bag (bag_ptr[j] = j, the one-hot
 * layout, grouped table by table): another layout with that count sets
 * HL_DEVERR_SHAPE; in that layout a hot code that names a row of another
 * table than its bag's (hl_remap's codes never do) sets HL_DEVERR_BAD_CODE
 * and is skipped. */
hl_status hl_embbag_bwd_sgd(hl_handle* h, void* w_hot, void* staging, int32_t staging_rows,
                            const int32_t* codes, const int32_t* bag_ptr, int32_t n_samples,
                            int32_t bags_per_sample, int64_t n_lookups, const int32_t* sample_ids,
                            const int32_t* n_sel_dev, int32_t n_sel_max, const float* dY, float lr,
                            void* workspace, size_t ws_bytes, hl_stream stream);

/* hl_embbag_bwd_sgd for callers that cannot allocate device memory (code under
 * graph capture, tight serving loops, harnesses that forbid allocation): the
 * same arguments but the workspace, the same updates bit for bit (same
 * kernels, same grouping).  The workspace is a file-scope device array of
 * hl_noalloc_scratch_bytes() = 32 MiB in the library, one copy per GPU, held
 * until the process ends (hl_create looks up its address on the handle's
 * device and zero-fills it once).  The call allocates nothing.  Mini-batches
 * whose plan needs more than the array (about 50 bytes per lookup at dim 64,
 * 85 at dim 128: each of the benchmark's mini-batches fits) return HL_ERR_CAPACITY and enqueue nothing.  Every call
 * on one GPU shares that GPU's array and leaves its last contents there: calls
 * that overlap on one GPU (on concurrent streams or host threads) race and
 * must not be issued. */
size_t hl_noalloc_scratch_bytes(void);
hl_status hl_embbag_bwd_sgd_noalloc(hl_handle* h, void* w_hot, void* staging, int32_t staging_rows,
                                    const int32_t* codes, const int32_t* bag_ptr, int32_t n_samples,
                                    int32_t bags_per_sample, int64_t n_lookups, const int32_t* sample_ids,
                                    const int32_t* n_sel_dev, int32_t n_sel_max, const float* dY, float lr,
                                    hl_stream stream);

/* The two halves of hl_embbag_bwd_sgd.  hl_embbag_bwd_plan groups the
 * selected lookups by code (it reads codes and bag_ptr only, not the rows or
 * dY) and leaves the grouping in the workspace; hl_embbag_bwd_apply reduces dY
 * over each group and updates the rows.  The plan can therefore run while the
 * working parameters are still being fetched and the forwards still read the
 * rows; the apply must come after both forwards (they read the pre-update
 * rows, Sec. IV-A Eq. 5) and after the fetch.  The apply takes the plan's
 * staging_rows, n_samples, bags_per_sample and n_lookups and the same
 * workspace, with no other call on that workspace in between; otherwise it
 * returns HL_ERR_INVALID_ARG and changes nothing.  Applying one plan twice is
 * two SGD steps with the same grouping. */
hl_status hl_embbag_bwd_plan(hl_handle* h, int32_t staging_rows, const int32_t* codes,
                             const int32_t* bag_ptr, int32_t n_samples, int32_t bags_per_sample,
                             int64_t n_lookups, const int32_t* sample_ids, const int32_t* n_sel_dev,
                             int32_t n_sel_max, void* workspace, size_t ws_bytes, hl_stream stream);
hl_status hl_embbag_bwd_apply(hl_handle* h, void* w_hot, void* staging, int32_t staging_rows,
                              int32_t n_samples, int32_t bags_per_sample, int64_t n_lookups,
                              const float* dY, float lr, void* workspace, size_t ws_bytes,
                              hl_stream stream);

/* hl_embbag_fwd over every sample followed by hl_embbag_bwd_plan over every
 * sample, with the same results (out bit for bit, the same grouping left in
 * the workspace for hl_embbag_bwd_apply).  The backward's grouping reads only
 * the codes (Sec. IV: hot rows are updated on the GPU after both forwards),
 * so for a one-hot mini-batch (one lookup per bag, grouped table by table)
 * the sorts of the tables run in the forward's launch, on compute units the
 * forward leaves free; other mini-batches take the two calls in turn.
 * Arguments as those two calls; the workspace as hl_embbag_bwd_plan's. */
hl_status hl_embbag_fwd_plan(hl_handle* h, const void* w_hot, const void* staging, int32_t staging_rows,
                             const int32_t* codes, const int32_t* bag_ptr, int32_t n_samples,
                             int32_t bags_per_sample, int64_t n_lookups, float* out, void* workspace,
                             size_t ws_bytes, hl_stream stream);

/* The grouping the last hl_embbag_bwd_plan left in `workspace` (with the same
 * staging_rows, n_samples, bags_per_sample and n_lookups; else
 * HL_ERR_INVALID_ARG), copied for inspection to keys_out and bags_out (device,
 * n_lookups entries each): one (key, bag) pair per lookup in the order the
 * reduction takes them, key = hot slot, or n_hot + staging row, or 0xFFFFFFFF
 * for a lookup the plan skipped.  The pairs of one key are contiguous and in
 * ascending lookup (CSR) order, hot keys come first, and the summation order of
 * the update (Sec. IV-A, Eq. 5: one coalesced step) follows this order. */
hl_status hl_embbag_bwd_grouping(hl_handle* h, int32_t staging_rows, int32_t n_samples, int32_t bags_per_sample,
                                 int64_t n_lookups, const void* workspace, size_t ws_bytes, uint32_t* keys_out,
                                 uint32_t* bags_out, hl_stream stream);

/* hl_embbag_bwd_apply in halves, bit for bit the same updates: part 1 reduces
 * dY for every group, updates the hot rows and keeps the sums of the staging
 * rows below n_lookups in the workspace without reading those rows (so it can
 * run while they are fetched, once the forwards have read the hot rows);
 * part 2 updates those staging rows from the kept sums (reads no dY).  Part 2
 * needs part 1 on the same plan (else HL_ERR_INVALID_ARG); part 0 is both. */
hl_status hl_embbag_bwd_apply_part(hl_handle* h, void* w_hot, void* staging, int32_t staging_rows,
                                   int32_t n_samples, int32_t bags_per_sample, int64_t n_lookups,
                                   const float* dY, float lr, int32_t part, void* workspace,
                                   size_t ws_bytes, hl_stream stream);

/* For tests of the sorts' fallback: the backward's grouping ranks the items
 * of each radix pass by equal keys, checks the pass kept the order of equal
 * digits and redoes it with ranks that are stable by construction (ballot
 * peer masks) if not; on != 0 makes every pass take the second form directly.
 * The grouping is the same either way. */
hl_status hl_debug_ballot_ranks(hl_handle* h, int32_t on);

/* ----------------------------------------------------------------- errors --
 * Waits for the device, returns the error word (HL_DEVERR_* bits) in *err_out
 * (host) and clears it.  Returns HL_ERR_DEVICE if any bit was set. */
hl_status hl_last_device_error(hl_handle* h, uint32_t* err_out);

/* ---------------------------------------------------------------- tracing --
 * Per-kernel timing with HIP events.  hl_trace_enable(h, cap) creates cap
 * event pairs, and every kernel the handle's calls launch (until cap records
 * exist) is launched so that its dispatch records the pair at its own start
 * and end (no marker packets on the stream); cap = 0 turns tracing off.
 * hl_trace_read waits for record i and returns its kernel name (static
 * string) and duration in ms; hl_trace_read_at also gives its start in ms
 * after record 0's start (records on several streams on one time line).
 * hl_trace_reset forgets the records.  hl_trace_only(h, names) records only
 * kernels of those comma-separated names, at most 255 characters (NULL: all
 * again); tracing every kernel of a pipelined step changes its schedule (the
 * traced launches take longer to issue), so a few names at a time. */
hl_status hl_trace_enable(hl_handle* h, int32_t cap);
hl_status hl_trace_only(hl_handle* h, const char* name);
int32_t hl_trace_count(const hl_handle* h);
hl_status hl_trace_read(const hl_handle* h, int32_t i, const char** name, float* ms);
hl_status hl_trace_read_at(const hl_handle* h, int32_t i, const char** name, float* start_ms, float* ms);
hl_status hl_trace_reset(hl_handle* h);

/* ---------------------------------------------------------------- streams --
 * A stream of default priority whose kernels run only on compute units
 * [first_cu, first_cu + n_cu) of the current device (complement != 0: on all
 * the others; n_cu = 0: no restriction).  The host-link copy keeps its compute
 * units' memory queues full of slow host reads, which stalls any kernel that
 * shares those units, so the pipelined schedule gives the copy a few units of
 * its own and the rest of the step the others. */
hl_status hl_stream_create(int32_t first_cu, int32_t n_cu, int32_t complement, hl_stream* out);
hl_status hl_stream_destroy(hl_stream stream);

/* --------------------------------------------------------------- pipeline --
 * The pipelined schedule of one mini-batch (Sec. IV and the pipeline figure:
 * the popular mu-batch runs on the GPU while the non-popular mu-batch's working
 * parameters are gathered), enqueued by one host call on three streams of the
 * pipeline's own: the host-link copy on compute units [0, fetch_cus) (0 = no
 * restriction), everything else on the other units.  The step runs
 * hl_dispatch, hl_cold_plan (no sample list: a cold lookup makes its sample
 * non-popular), hl_cold_fetch beside hl_embbag_fwd_part 1 over every sample
 * (the popular mu-batch's forward and the non-popular one's hot half in one
 * launch: the same sums), hl_embbag_bwd_plan and apply part 1 on a third
 * stream, then part 2 of the forward over the non-popular mu-batch and of the
 * apply (and with write_back, hl_cold_scatter after the updates).  It is ordered after the work already on `stream`, and
 * `stream` waits for it (the write-back excepted: it is ordered before the
 * next step's fetch and before any later step's plan that rewrites the same
 * cold_ids, so callers that write back may alternate two cold_ids / n_cold
 * buffers between steps; hl_pipeline_sync_writeback makes `stream` wait for
 * the last write-backs).
 * One pipeline serves one handle; steps on it do not overlap other calls on
 * the same workspace.  Every buffer keeps the meaning it has in the calls
 * above; counts has 2 entries.  Refused (HL_ERR_UNSUPPORTED) while `stream` is
 * being captured into a graph: a graph keeps no stream's compute-unit mask. */
typedef struct hl_pipeline hl_pipeline;
typedef struct hl_step_io {
  const uint32_t* rows;       /* mini-batch (device) */
  const int32_t* bag_ptr;
  int32_t n_samples;
  int32_t bags_per_sample;
  int64_t n_lookups;
  const float* dY;            /* NULL: forward only */
  float lr;
  uint32_t* gids;             /* per-step results (device) */
  int32_t* codes;
  uint8_t* flags;
  int32_t* pop_ids;
  int32_t* nonpop_ids;
  int32_t* counts;
  uint32_t* cold_ids;
  int32_t* n_cold;
  const void* w_host;         /* parameters */
  void* w_hot;
  void* staging;
  int32_t staging_cap;
  float* out;
  void* workspace;
  size_t ws_bytes;
  int32_t write_back;
  uint32_t step_flags;        /* HL_STEP_* */
} hl_step_io;
/* Step flag: no ordering with `stream` (no wait before, no wait after); the
 * caller has the inputs ready on the device and later calls
 * hl_pipeline_sync.  Back-to-back steps then run without two cross-stream
 * hops per step. */
#define HL_STEP_UNTIED 1u
/* Step flag: the step's hl_dispatch and hl_cold_plan were enqueued ahead by
 * hl_pipeline_plan with the same inputs, sizes and per-step buffers (gids,
 * codes, flags, pop_ids, nonpop_ids, counts, cold_ids, n_cold, workspace);
 * the step skips them.  HL_ERR_INVALID_ARG if no such plan is pending. */
#define HL_STEP_PLANNED 2u
/* Step flag (also read by hl_pipeline_plan): the waits of the handovers
 * between the pipeline's streams run in kernels of their own, launched around
 * the calls, instead of inside the path's kernels (whose first block otherwise
 * waits as the kernel ends, or every block as it starts).  Same order, same
 * results, a few more launches; the path's kernels then hold no waits, so
 * their durations are their own work (for timing them in the pipelined
 * schedule). */
#define HL_STEP_HANDOVER_KERNELS 4u
/* fetch_cus compute units [0, fetch_cus) run the host-link copy (0: no masks
 * at all); plan_cus > 0 gives the look-ahead plans the next plan_cus units of
 * their own (0: they share main's).  Masks in multiples of 8 units keep every
 * XCD equally loaded (plans on 56 or 48 units measured 35% slower steps); fetch
 * 8, plan 64, main the other 184 measured fastest here.  The runtime refuses
 * masks of fewer than 8 units.  With masks the streams hand over through
 * device flags, which needs each stream on a hardware queue of its own: the
 * call checks every pair that hands over (a bounded wait enqueued ahead of its
 * signal, ~10 ms at most) and returns HL_ERR_UNSUPPORTED if one ran out. */
hl_status hl_pipeline_create(hl_handle* h, int32_t fetch_cus, int32_t plan_cus, hl_pipeline** out);
hl_status hl_pipeline_destroy(hl_pipeline* p);
hl_status hl_pipeline_step(hl_pipeline* p, const hl_step_io* io, hl_stream stream);
/* Look-ahead segregation (Sec. IV and the pipeline figure: the accelerator
 * classifies and segregates a mini-batch while the GPUs train the one before):
 * enqueues hl_dispatch, hl_cold_plan and, when io->dY is not NULL,
 * hl_embbag_bwd_plan of io's mini-batch on a fourth stream of the pipeline, to
 * be consumed by a later hl_pipeline_step with HL_STEP_PLANNED and the same io
 * (dY NULL or not alike).  The plan waits for every step enqueued before it
 * that used one of its per-step buffers (gids, codes, flags, pop_ids,
 * nonpop_ids, counts, cold_ids, n_cold) or its workspace, which it rewrites,
 * for every step enqueued before it that ran its own dispatch (the cold-gather
 * hash table is shared), and for the write-back that last read its cold_ids;
 * one step ahead thus needs two sets of per-step buffers, alternated, and
 * enqueuing a step before the plan of the batch after it lets the plan run
 * beside that step.  The planned step's row fetch still waits for the last
 * step that used its staging rows to end, and its forwards and backward run on
 * one stream.  lr, w_host, w_hot, staging, out and
 * write_back are not read.  HL_STEP_UNTIED in io->step_flags: no wait for
 * `stream` first.  HL_ERR_INVALID_ARG: a plan on the same workspace is still
 * pending, or four plans are; HL_ERR_UNSUPPORTED: a pipeline without
 * compute-unit masks (fetch_cus = 0), whose streams may share hardware queues,
 * or `stream` under capture. */
hl_status hl_pipeline_plan(hl_pipeline* p, const hl_step_io* io, hl_stream stream);
hl_status hl_pipeline_sync_writeback(hl_pipeline* p, hl_stream stream);
/* `stream` waits for every step and plan enqueued so far (and the write-backs). */
hl_status hl_pipeline_sync(hl_pipeline* p, hl_stream stream);
/* The pipeline's streams (main and group on the compute units the copy leaves
 * free, fetch on the copy's own), for callers that enqueue more work in the
 * same arrangement instead of creating streams of their own (a process has a
 * few hardware queues; streams beyond them share queues). */
hl_status hl_pipeline_streams(const hl_pipeline* p, hl_stream* main, hl_stream* fetch, hl_stream* group);

/* ---------------------------------------------------- pinned host memory --
 * Page-locked host memory mapped into the device address space (the host
 * table the cold gather reads).  *host receives the host pointer, *dev (may be
 * NULL) the pointer kernels use. */
hl_status hl_host_alloc(size_t bytes, void** host, void** dev);
hl_status hl_host_free(void* host);

#ifdef __cplusplus
}
#endif
#endif /* HOTLINE_H */
