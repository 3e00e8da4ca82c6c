/*
 * moe.h -- C ABI of libmoe: the MoE dispatch/combine hot path on one MI355X.
 *
 * The operator follows the paper's MoE dispatch/combine (Section 8.1 and
 * Table 2) and the hierarchical workload partitioning it is built on
 * (Appendix D): token placement (per-expert counts, prefix-sum offsets and
 * token-local offsets), expert windows grouped per peer into peer windows,
 * and a byte-balanced split of the copy work over the GPU's workgroups
 * (Section 6.2).  The R destination peers ("ranks") of expert parallelism are
 * emulated as R separate receive regions in the same GPU's HBM, addressed
 * through a device-side table of region base addresses; this table plays the
 * role of the per-peer destination addresses of the remote-slice tuple
 * <peer, src, dst, bytes, op, flag> of Section 6.1.
 *
 * Shapes and notation: T tokens, hidden size H, k routed slots per token,
 * E experts spread over R ranks in contiguous blocks of L = E/R (expert e
 * lives on rank e / L).  topk_idx[T,k] int32 holds the expert of each slot
 * (-1 = unused slot), topk_w[T,k] float32 its combine weight.  One routed row
 * exists per (token, expert) pair; rows are ordered by (expert, token), so
 * the rows of rank r are the global rows [rank_offset[r], rank_offset[r+1])
 * and land in region r at region-local row (global row - rank_offset[r]).
 *
 * Conventions for every entry point:
 *  - All array arguments are DEVICE pointers unless marked "host".  The
 *    caller allocates and owns every buffer; the library allocates, frees
 *    and caches no memory (moe_layout_scratch uses one fixed array of the
 *    library's, see there).  Host-side it keeps only what it reads once per
 *    device (device properties, that array's address).  Device-side, the
 *    default work split of moe_dispatch / moe_combine hands parts out from
 *    ticket counters in the caller's workspace, which every call leaves at
 *    zero: calls that share a workspace must not overlap in time; separate
 *    workspaces are independent.
 *  - `stream` is a hipStream_t passed as void* (NULL = the null stream).
 *    Every call only enqueues kernels on `stream` and returns without
 *    synchronizing; outputs are ready when the stream reaches that point.
 *  - Return codes (host side, checked before anything is enqueued; on error
 *    nothing is launched): MOE_OK, MOE_EINVAL (null pointer where one is
 *    required, T < 0, k < 1, k > MOE_MAX_K, k > E, E % R != 0,
 *    E > MOE_MAX_EXPERTS, T*k > INT32_MAX, H < 1, a row of more than
 *    INT32_MAX bytes, bad dtype), MOE_EALIGN (x
 *    or y not 16-byte aligned, row bytes not a multiple of 16, fp8 H not a
 *    multiple of 128, x_scales not 4-byte aligned; region base addresses sit
 *    in device tables and their alignment is the caller's to keep),
 *    MOE_EWORKSPACE (workspace too small or not 256-byte aligned),
 *    MOE_ELAUNCH (a HIP launch failed; moe_last_hip_error() has the code).
 *  - Device status word `status` (uint32, device): the caller zeroes it;
 *    kernels OR these bits into it and the caller reads it whenever it
 *    synchronizes: MOE_STATUS_BAD_INDEX (an index outside [-1, E): the slot
 *    is treated as unused; the copy kernels also set it for a slot whose pos
 *    is set but whose index names no rank -- pos does not belong to
 *    topk_idx -- and skip that slot), MOE_STATUS_DUP_INDEX (an expert repeated within
 *    one token's row: later repeats are treated as unused),
 *    MOE_STATUS_CAPACITY (a row's region-local index is outside
 *    [0, recv_cap[r]): dispatch does not write it and combine does not read
 *    it; a negative index only arises when pos does not belong to topk_idx),
 *    MOE_STATUS_LAYOUT_SYNC (the layout's workgroups did not all reach its
 *    grid barrier within 2 s -- other work held the compute units that long;
 *    that call's outputs are not valid: the chunks whose workgroups gave up
 *    waiting leave their slots unrouted (pos = -1) and parts of the plan
 *    unwritten, and dispatch and combine still stay inside their buffers --
 *    they clamp plan ranges to the batch and skip slots whose rank is out of
 *    range.  The environment variable MOE_LAYOUT_SYNC_LIMIT_US, read once
 *    per device, replaces the 2 s limit; tests use it to reach this path).
 *  - The three calls of one batch must see the same topk_idx, T, k, E, R and
 *    workspace; dispatch and combine read the partition plan that moe_layout
 *    leaves in the workspace.
 */
#ifndef MOE_H_
#define MOE_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define MOE_VERSION 5

#define MOE_OK 0
#define MOE_EINVAL (-1)
#define MOE_EALIGN (-2)
#define MOE_EWORKSPACE (-3)
#define MOE_ELAUNCH (-4)

#define MOE_DTYPE_BF16 0     /* hidden rows of H bf16 values (2H bytes) */
#define MOE_DTYPE_FP8_E4M3 1 /* H OCP E4M3FN bytes + H/128 float32 block scales */

#define MOE_STATUS_BAD_INDEX 1u
#define MOE_STATUS_DUP_INDEX 2u
#define MOE_STATUS_CAPACITY 4u
#define MOE_STATUS_LAYOUT_SYNC 8u

#define MOE_MAX_K 32
#define MOE_MAX_EXPERTS 1024
#define MOE_FP8_BLOCK 128

/* Number of parts P of the byte-balanced partition plan (parts of equal byte
 * cost).  moe_dispatch and moe_combine launch W wavefronts, W a power of
 * two that divides P (dispatch 256 to 4096, combine 512 to 4096, sized from
 * the bytes each wavefront keeps in flight).  Wavefront g starts at part g;
 * later parts are either strided statically (g+W, g+2W, ...) or handed out
 * at run time in plan order, as MOE_POLICY_BALANCED describes.
 * 12288 = 3 * 2^12 also divides evenly over 256 compute units at 4, 8, 12,
 * 16, 24 or 48 wavefronts each. */
#define MOE_PLAN_PARTS 12288

/* Library version (MOE_VERSION). */
int moe_version(void);

/* Static, human-readable text for a return code. */
const char* moe_strerror(int code);

/* The hipError_t of the last failed launch on the calling thread (0 if
 * none). */
int moe_last_hip_error(void);

/* Rate of the clock the trace buffers of moe_dispatch_ex / moe_combine_ex
 * use on the current device, in kHz (written to *khz, a HOST pointer). */
int moe_wall_clock_khz(int* khz);

/*
 * moe_layout_workspace_bytes -- device workspace that moe_layout needs for
 * a batch of this shape (written to *out_bytes, a HOST pointer).  The
 * workspace starts with the partition plan: int32 bound[MOE_PLAN_PARTS + 1],
 * token boundaries of the parts (part p = tokens [bound[p], bound[p+1])).
 * The rest is scratch whose content is internal.
 */
int moe_layout_workspace_bytes(int64_t T, int k, int E, int R, size_t* out_bytes);

/*
 * moe_layout -- token placement (Appendix D, first level: destination
 * expert, per-expert counts, prefix-sum offsets and token-local offsets;
 * second and third level: expert windows and the peer windows they form)
 * plus the byte-balanced partition plan (Section 6.2, one memory tier).
 *
 * In:  topk_idx [T,k] int32 row-major.
 * Out: expert_count[E]      routed slots per expert;
 *      expert_offset[E+1]   exclusive prefix sum of expert_count
 *                           (expert_offset[E] = number of routed slots N);
 *      rank_count[R]        routed slots per rank (peer window sizes, rows);
 *      rank_offset[R+1]     rank_offset[r] = expert_offset[r*L], [R] = N;
 *      pos[T*k]             global row of slot (t,j), -1 if unused: rows are
 *                           ordered by (expert, token), so
 *                           pos = expert_offset[e] + #{t' < t routed to e};
 *      row_src[T*k]         inverse map: slot index t*k+j of global row i for
 *                           i < N, -1 for i >= N;
 *      workspace            partition plan (see above) + scratch;
 *      status               OR-ed bits (BAD_INDEX, DUP_INDEX, LAYOUT_SYNC).
 * Launches: one workgroup when T <= 256; one launch whose workgroups (one
 * per 256-token chunk, at most 128) meet at a grid barrier when the batch
 * fits that; a counting launch and a placing launch otherwise.  The barrier
 * needs no cleared memory: the workspace holds a generation word that each
 * such call advances on the device, and a workgroup's arrival flag carries a
 * 64-bit hash of it, which leftover memory matches only by chance (2^-64).
 * The workspace may therefore be uninitialised, reused across shapes, or
 * used from a replayed graph.
 * Results are deterministic and bit-identical from run to run.  T = 0 is
 * allowed (counts and offsets become 0).
 */
int moe_layout(const int32_t* topk_idx, int64_t T, int k, int E, int R,
               int32_t* expert_count, int32_t* expert_offset, int32_t* rank_count,
               int32_t* rank_offset, int32_t* pos, int32_t* row_src, void* workspace,
               size_t workspace_bytes, uint32_t* status, void* stream);

/*
 * moe_layout_scratch -- moe_layout for callers that cannot allocate device
 * memory (code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc): the same kernels and the same outputs, but the
 * workspace is the library's own, a fixed device array of 576 KiB per GPU
 * (held until the process ends), large enough for every shape the library
 * accepts (moe_layout_workspace_bytes never exceeds 581888 bytes).  This
 * call allocates and frees nothing.
 *
 * In/out: as moe_layout, without the workspace arguments.
 * workspace        HOST out: device address of the library's workspace on
 *                  the current device; pass it, with *workspace_bytes, as
 *                  the workspace of this batch's moe_dispatch / moe_combine
 *                  (and moe_dispatch_ex, moe_combine_ex).  Its front holds
 *                  the partition plan, as for moe_layout.
 * workspace_bytes  HOST out: moe_layout_workspace_bytes for this shape.
 * Every call on one GPU uses that GPU's one array and leaves its plan there
 * until the next call: the batch's dispatch and combine must be enqueued
 * before the next moe_layout_scratch on that GPU, and calls (this one, or
 * the dispatch / combine that use its workspace) that overlap on one GPU --
 * concurrent streams, other host threads -- race.  The first call on a
 * device looks the array's address up (hipGetSymbolAddress); make that
 * first call outside graph capture.
 * Errors: as moe_layout (argument errors are found before any HIP call);
 * MOE_EINVAL for null workspace / workspace_bytes; MOE_EWORKSPACE if a
 * shape needed more than the array (none does); MOE_ELAUNCH if the address
 * lookup fails.
 */
int moe_layout_scratch(const int32_t* topk_idx, int64_t T, int k, int E, int R,
                       int32_t* expert_count, int32_t* expert_offset, int32_t* rank_count,
                       int32_t* rank_offset, int32_t* pos, int32_t* row_src, uint32_t* status,
                       void** workspace, size_t* workspace_bytes, void* stream);

/*
 * moe_layout_fixed -- token placement into fixed-capacity expert windows:
 * the low-latency form of the operator (Table 2's LL rows; the paper does
 * not define the mode, this is the reading taken).  Expert e owns global rows
 * [e*capacity, (e+1)*capacity), so every offset is known before routing and
 * receive regions of L*capacity rows per rank can be allocated once; no host
 * read of the counts is needed between layout and dispatch, and the whole
 * layout -> dispatch -> combine chain can run inside one captured graph.
 * Within a window rows are in token order; a routed slot whose rank within
 * its expert reaches `capacity` is dropped (pos = -1, MOE_STATUS_CAPACITY).
 *
 * Out: expert_count[E] = rows placed per expert (<= capacity);
 *      expert_offset[e] = e*capacity (E+1 entries);
 *      rank_count[R] = rows placed per rank; rank_offset[r] = r*L*capacity;
 *      pos[T*k] as moe_layout; row_src[E*capacity]: slot of each window row,
 *      -1 for rows no slot fills; the partition plan counts placed slots.
 * Dispatch and combine take these outputs unchanged (recv_cap[r] = L*capacity
 * for regions sized to whole windows).  Errors as moe_layout, plus
 * MOE_EINVAL for capacity < 0 or E*capacity > INT32_MAX.
 */
int moe_layout_fixed(const int32_t* topk_idx, int64_t T, int k, int E, int R, int capacity,
                     int32_t* expert_count, int32_t* expert_offset, int32_t* rank_count,
                     int32_t* rank_offset, int32_t* pos, int32_t* row_src, void* workspace,
                     size_t workspace_bytes, uint32_t* status, void* stream);

/*
 * moe_dispatch -- copy every routed token row to its destination rank's
 * receive region (Section 6.1 remote-slice transfers with op = store, one
 * per routed slot; work split over wavefronts by bytes, Section 6.2 and
 * Appendix D third level).  A pure byte copy: for each routed slot (t,j)
 * with expert e, rank r = e/L and local = pos[t*k+j] - rank_offset[r] <
 * recv_cap[r]:
 *      region_r[local, :] = x[t, :]                       (row_bytes)
 *      scale_region_r[local, :] = x_scales[t, :]          (fp8 only)
 *
 * x         [T,H] bf16 (dtype BF16) or [T,H] E4M3FN bytes (dtype FP8_E4M3),
 *           16-byte aligned; row bytes = 2H or H, a multiple of 16.
 * x_scales  [T,H/128] float32 for FP8_E4M3, else NULL.
 * recv_x    [R] uint64 region base addresses (device table), 16-byte aligned;
 *           region r holds recv_cap[r] rows of row_bytes each.
 * recv_scales [R] uint64 scale-region bases (FP8_E4M3) or NULL; region r
 *           holds recv_cap[r] rows spaced scale_pitch bytes apart.
 * scale_pitch bytes from one scale row to the next in a scale region; 0
 *           means packed rows of (H/128)*4 bytes.  Otherwise at least
 *           (H/128)*4 and a multiple of 4.  Dispatch writes the whole pitch:
 *           the row's scales, then zeros.  A pitch that is a multiple of 128
 *           (with 128-byte aligned region bases) gives every scale row its
 *           own cache lines, so no two rows share a line that different
 *           wavefronts write partially; packed 224-byte rows cost ~30 us more
 *           per 131k rows on MI355X.
 * recv_cap  [R] int32 capacity of each region in rows.
 * topk_idx, pos, rank_offset, workspace: as produced by moe_layout.  Parts
 *           of the plan are handed out at run time from a counter in the
 *           workspace (all but each wavefront's first when parts carry 64
 *           KiB or more, else the second half; MOE_POLICY_BALANCED of
 *           moe_dispatch_ex): two dispatch calls that share a workspace must
 *           not run at the same time on different streams.
 * Bytes of a region beyond the rows dispatch writes are left untouched.
 */
int moe_dispatch(const void* x, const float* x_scales, int dtype, int64_t T, int H,
                 int k, int E, int R, const int32_t* topk_idx, const int32_t* pos,
                 const int32_t* rank_offset, const uint64_t* recv_x,
                 const uint64_t* recv_scales, int scale_pitch, const int32_t* recv_cap,
                 const void* workspace, size_t workspace_bytes, uint32_t* status,
                 void* stream);

/* Work-split policies of moe_dispatch_ex / moe_combine_ex (all give
 * bit-identical regions and identical y). */
#define MOE_POLICY_BALANCED 0 /* byte-balanced parts, the library's choice: when a
                               * part carries 64 KiB (dispatch) or 128 KiB (combine)
                               * or more on average, every part after each
                               * wavefront's first is handed out at run time;
                               * smaller parts: dispatch assigns the first half
                               * statically and hands the rest out at run time (all
                               * statically when a wavefront would own fewer than 8
                               * parts), combine assigns all statically
                               * (moe_dispatch, moe_combine) */
#define MOE_POLICY_ROWS 1     /* pull: the N routed rows split evenly over wavefronts */
#define MOE_POLICY_BY_RANK 2  /* pull: a fixed group of W/R wavefronts per rank */
#define MOE_POLICY_DYNAMIC 3  /* push; every part after the first handed out at run time */
#define MOE_POLICY_STATIC 4   /* push; every part assigned statically (parts g, g+W, ...) */

/*
 * moe_dispatch_ex -- moe_dispatch with a choice of work split and an
 * optional per-wavefront trace; for studying the partitioning of Section 6.2
 * (Section 9.6 compares a naive per-peer core assignment with the balanced
 * one; MOE_POLICY_BY_RANK is that naive assignment, MOE_POLICY_ROWS splits
 * the same pull work evenly, MOE_POLICY_BALANCED is the product path).
 *
 * policy       one of MOE_POLICY_*; anything else is MOE_EINVAL.  Parts
 *              handed out at run time (MOE_POLICY_DYNAMIC, and under
 *              MOE_POLICY_BALANCED all of them for large parts or the second
 *              half of dispatch's for small ones) are claimed in plan order
 *              from a counter in the workspace (moe_layout zeroes it; the
 *              last wavefront of a launch resets it), so faster wavefronts
 *              take more parts.  Dispatch calls that share a workspace must
 *              therefore not run concurrently under these policies, nor
 *              combine calls (dispatch and combine use separate counters);
 *              calls one after another on a stream, or replayed in a graph,
 *              are fine.
 * waves        wavefronts to launch: 0 lets the library choose (the product
 *              choice; the push policies use the count of moe_dispatch, the
 *              pull policies as many as the device holds at once); otherwise
 *              a multiple of 4 that
 *              divides MOE_PLAN_PARTS (and, under MOE_POLICY_BY_RANK, a
 *              multiple of R), else MOE_EINVAL.  Fewer wavefronts occupy fewer
 *              compute units: sweeping the count shows how each split's
 *              balance depends on the number of cores sharing the work.
 * trace        NULL, or a device buffer of 2*trace_waves uint64: wavefront g
 *              (g < trace_waves) writes trace[2g] = its start time and
 *              trace[2g+1] = the time its last store completed, both from the
 *              GPU's constant-rate wall clock (hipDeviceAttributeWallClockRate
 *              kHz).  The launch uses at most MOE_PLAN_PARTS wavefronts;
 *              entries of wavefronts that do not exist are left untouched.
 * Other arguments, results and errors are those of moe_dispatch.
 */
int moe_dispatch_ex(const void* x, const float* x_scales, int dtype, int64_t T, int H,
                    int k, int E, int R, const int32_t* topk_idx, const int32_t* pos,
                    const int32_t* rank_offset, const int32_t* row_src, const uint64_t* recv_x,
                    const uint64_t* recv_scales, int scale_pitch, const int32_t* recv_cap,
                    const void* workspace, size_t workspace_bytes, uint32_t* status,
                    int policy, int waves, uint64_t* trace, int trace_waves, void* stream);

/*
 * moe_combine -- gather each token's expert outputs back to token order and
 * reduce them with the top-k weights (Section 6.1: operands are loaded and
 * accumulated on chip, then written once; token-centric, so no two
 * wavefronts write the same output row and no atomics are needed):
 *      y[t, :] = bf16( sum over routed slots j of topk_w[t,j] * Y_r[local, :] )
 * with r, local as in moe_dispatch and Y_r the bf16 expert-output region of
 * rank r (expert_y[r], rows of 2H bytes).  Products and the sum are float32,
 * the result is rounded to bf16 to nearest-even.  A token with no routed
 * slot gets +0.  Slots whose local row reaches recv_cap[r] are skipped.
 *
 * expert_y  [R] uint64 bf16 region bases (device table), 16-byte aligned.
 * topk_w    [T,k] float32.
 * y         [T,H] bf16 output, 16-byte aligned, 2H a multiple of 16.
 * workspace as produced by moe_layout.  When parts carry 128 KiB or more,
 *           all but each wavefront's first are handed out at run time from
 *           a counter in the workspace (separate from dispatch's): two
 *           combine calls that share a workspace must not run at the same
 *           time on different streams.
 */
int moe_combine(const uint64_t* expert_y, const float* topk_w, int64_t T, int H, int k,
                int E, int R, const int32_t* topk_idx, const int32_t* pos,
                const int32_t* rank_offset, const int32_t* recv_cap, uint16_t* y,
                const void* workspace, size_t workspace_bytes, uint32_t* status,
                void* stream);

/*
 * moe_combine_ex -- moe_combine with a work split (MOE_POLICY_BALANCED and
 * MOE_POLICY_STATIC: all parts assigned statically; MOE_POLICY_DYNAMIC as
 * for moe_dispatch_ex; others are MOE_EINVAL), the
 * wavefront count and the optional per-wavefront trace of moe_dispatch_ex
 * (same rules, layout and clock).
 */
int moe_combine_ex(const uint64_t* expert_y, const float* topk_w, int64_t T, int H, int k,
                   int E, int R, const int32_t* topk_idx, const int32_t* pos,
                   const int32_t* rank_offset, const int32_t* recv_cap, uint16_t* y,
                   const void* workspace, size_t workspace_bytes, uint32_t* status,
                   int policy, int waves, uint64_t* trace, int trace_waves, void* stream);

/* ------------------------------------------------------------------------
 * Per-peer deduplicated path.  A token with several experts on one rank is
 * sent to that rank once: one row per routed (token, rank) pair ("pair
 * row") instead of one per (token, expert) pair, so the bytes that cross to
 * each peer -- the per-peer payload B_p that the partitioning of Section 6.2
 * balances -- drop by the duplicates.  The receiving rank then rebuilds its
 * expert windows locally (moe_expand) and, on the way back, reduces each
 * pair's expert outputs to one partial row (moe_combine_local) that the
 * source adds up (moe_combine_dedup).  Appendix D's first level (placement)
 * and second level (expert windows) are unchanged; the peer windows of the
 * third level hold pair rows.
 *
 * Pair rows of rank r are the global pair rows [tok_offset[r],
 * tok_offset[r+1]), in token order, at region-local row (pair row -
 * tok_offset[r]) of that rank's pair region.  A slot's pair is (t, e/L); the
 * pair row is carried by the token's first routed slot on that rank.
 * ------------------------------------------------------------------------ */

/* Workspace bytes of moe_layout_dedup (written to *out_bytes, HOST).  Its
 * front holds the pair-row plan: int32 bound[MOE_PLAN_PARTS + 1] over
 * tokens, a token costing one row read plus one row per pair. */
int moe_layout_dedup_workspace_bytes(int64_t T, int k, int E, int R, size_t* out_bytes);

/*
 * moe_layout_dedup -- placement of pair rows.  Slots are routed under the
 * rules of moe_layout (unused, out-of-range and repeated experts are not;
 * status bits 1 and 2 as there).
 *
 * Out: tok_count[R]       tokens sent to rank r (pairs of rank r);
 *      tok_offset[R+1]    exclusive prefix sum of tok_count ([R] = pairs);
 *      tok_pos[T*k]       on the first routed slot of token t on rank r:
 *                         global pair row of (t, r) = tok_offset[r] +
 *                         #{t' < t with a routed slot on r}; -1 on all other
 *                         slots;
 *      tok_src[T*k]       slot index t*k+j carrying each pair row (first
 *                         tok_offset[R] entries; the rest are -1);
 *      workspace          pair-row plan (see above) plus internal scratch,
 *                         moe_layout_dedup_workspace_bytes, 256-byte aligned.
 * A separate workspace from moe_layout's: the per-slot calls (moe_expand,
 * moe_combine_local) read moe_layout's plan, the pair-row calls
 * (moe_dispatch_dedup, moe_combine_dedup) read this one.
 */
int moe_layout_dedup(const int32_t* topk_idx, int64_t T, int k, int E, int R, int32_t* tok_count,
                     int32_t* tok_offset, int32_t* tok_pos, int32_t* tok_src, void* workspace,
                     size_t workspace_bytes, uint32_t* status, void* stream);

/*
 * moe_dispatch_dedup -- copy each pair row once: x[t] (and its fp8 scale
 * row) to region r at local row tok_pos - tok_offset[r] for every slot with
 * tok_pos >= 0 (Section 6.1 transfers, one per pair).  Arguments, layout,
 * alignment and errors are those of moe_dispatch with (tok_pos, tok_offset)
 * in place of (pos, rank_offset), regions sized in pair rows (recv_cap[r] >=
 * tok_count[r] to keep every row) and the moe_layout_dedup workspace.
 */
int moe_dispatch_dedup(const void* x, const float* x_scales, int dtype, int64_t T, int H, int k,
                       int E, int R, const int32_t* topk_idx, const int32_t* tok_pos,
                       const int32_t* tok_offset, const uint64_t* recv_x,
                       const uint64_t* recv_scales, int scale_pitch, const int32_t* recv_cap,
                       const void* workspace, size_t workspace_bytes, uint32_t* status,
                       void* stream);

/*
 * moe_expand -- receiver side of the deduplicated dispatch: every routed
 * slot (t, j) with expert e on rank r gets its pair row, copied from pair
 * region r (local row pair row - tok_offset[r]) to expert-ordered region r
 * at local row pos[t,j] - rank_offset[r].  The expert regions end up byte
 * for byte as moe_dispatch leaves them (fp8 scale rows included, their
 * pitch padding zeroed); each pair row is read once and written once per
 * expert of the pair.
 *
 * dedup_x / dedup_scales / dedup_cap: pair regions as written by
 *     moe_dispatch_dedup (scale rows scale_pitch bytes apart in both);
 * recv_x / recv_scales / recv_cap: expert-ordered regions as for
 *     moe_dispatch;
 * pos, rank_offset, workspace: from moe_layout (its plan splits the work);
 * tok_pos, tok_offset: from moe_layout_dedup.
 * A pair row at or past dedup_cap[r], or a destination at or past
 * recv_cap[r], is skipped and sets MOE_STATUS_CAPACITY.  Other errors as
 * moe_dispatch.
 */
int moe_expand(const uint64_t* dedup_x, const uint64_t* dedup_scales, int dtype, int64_t T,
               int H, int k, int E, int R, const int32_t* topk_idx, const int32_t* pos,
               const int32_t* rank_offset, const int32_t* tok_pos, const int32_t* tok_offset,
               const int32_t* dedup_cap, const uint64_t* recv_x, const uint64_t* recv_scales,
               int scale_pitch, const int32_t* recv_cap, const void* workspace,
               size_t workspace_bytes, uint32_t* status, void* stream);

/*
 * moe_combine_local -- receiver side of the deduplicated combine: for every
 * pair (t, r), the weighted sum of the token's expert outputs on rank r,
 *      partial_r[q - tok_offset[r], :] = bf16( sum over routed slots j of
 *                 token t with expert on r of topk_w[t,j] * Y_r[local, :] )
 * (q the pair row; Y_r and local as in moe_combine; float32 products and
 * sums, one rounding to bf16 to nearest-even).  Section 6.1 reduces on chip
 * and writes once: each partial row has one writer.
 *
 * expert_y / recv_cap: bf16 expert-output regions (rows of 2H bytes);
 * partial / part_cap: [R] bf16 partial regions in pair rows, 16-byte aligned;
 * pos, rank_offset, workspace: from moe_layout; tok_pos, tok_offset: from
 * moe_layout_dedup.  Expert rows at or past recv_cap[r] are not summed,
 * pair rows at or past part_cap[r] are not written; both set
 * MOE_STATUS_CAPACITY.  Other errors as moe_combine.
 */
int moe_combine_local(const uint64_t* expert_y, const float* topk_w, int64_t T, int H, int k,
                      int E, int R, const int32_t* topk_idx, const int32_t* pos,
                      const int32_t* rank_offset, const int32_t* recv_cap,
                      const int32_t* tok_pos, const int32_t* tok_offset,
                      const int32_t* part_cap, const uint64_t* partial, const void* workspace,
                      size_t workspace_bytes, uint32_t* status, void* stream);

/*
 * moe_combine_dedup -- source side of the deduplicated combine:
 *      y[t, :] = bf16( sum over the token's pairs (t, r) of
 *                      partial_r[q - tok_offset[r], :] )
 * in float32, rounded once to bf16 (nearest-even); a token with no pair gets
 * +0.  Pair rows at or past part_cap[r] are skipped (MOE_STATUS_CAPACITY).
 * Since each partial is itself rounded to bf16, y carries up to one more
 * bf16 rounding per pair than moe_combine's result.  Workspace: from
 * moe_layout_dedup.  Other arguments and errors as moe_combine.
 */
int moe_combine_dedup(const uint64_t* partial, int64_t T, int H, int k, int E, int R,
                      const int32_t* topk_idx, const int32_t* tok_pos,
                      const int32_t* tok_offset, const int32_t* part_cap, uint16_t* y,
                      const void* workspace, size_t workspace_bytes, uint32_t* status,
                      void* stream);

/*
 * moe_expert_scale -- stand-in expert for tests and benchmarks, not part of
 * the operator: for every global row g < expert_offset[E] of expert e on
 * rank r with local = g - rank_offset[r] < recv_cap[r],
 *      out_r[local, h] = bf16( v * s_e ),  s_e = identity ? 1 : 1 + 0.01*e
 * where v = float(bf16 input) or (float(fp8 input) * block scale), every
 * step a separately rounded float32 operation (no fused multiply-add) and
 * the result rounded to bf16 to nearest-even.
 *
 * recv_x / recv_scales / scale_pitch: region tables as for moe_dispatch
 * (dtype selects the payload); out_y: [R] uint64 bf16 output regions (rows of
 * 2H bytes).
 * max_rows: an upper bound on expert_offset[E] (normally T*k).
 */
int moe_expert_scale(const uint64_t* recv_x, const uint64_t* recv_scales, int scale_pitch,
                     int dtype, int H, int E, int R, int identity,
                     const int32_t* expert_offset,
                     const int32_t* rank_offset, const int32_t* recv_cap,
                     const uint64_t* out_y, int64_t max_rows, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MOE_H_ */
