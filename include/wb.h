/*
 * wb.h -- C ABI of libwb, the MI355X (gfx950) resharding library for
 * trainer-to-rollout weight transfer (WeightBridge, arXiv 2609.25442).
 *
 * The library covers the data-parallel hot path of the paper's transfer:
 *   1. describe a side's layout as slice-copy placements (Sec. 3.1: a worker's
 *      source map is the sequence of slice copies, each optionally transposed,
 *      that its weight loader performs from the full checkpoint);
 *   2. plan (Sec. 3.2, "Generating an efficient routing plan"): intersect trainer
 *      and rollout source maps in the checkpoint index space, give every needed
 *      element exactly one sender, split replicated tensors into distinct
 *      slices so the trainers send one copy, and balance bytes over replicas;
 *   3. pack (Sec. 3.2, packing kernel): coalesce one trainer rank's shards, in
 *      checkpoint row-major order, into one contiguous region per receiver;
 *   4. unpack (Sec. 3.2, assembly kernel): scatter the received regions into
 *      one rollout rank's tensors, casting fp32 -> bf16 (round to nearest
 *      even) or quantising to fp8 E4M3FN with 128x128 blockwise fp32 scales
 *      (s = amax / 448, q = RNE(x / s)); the paper assumes matched precision
 *      and names conversion as future work (Sec. 5).
 *
 * Conventions for every call:
 *   - Return value: WB_OK (0) or a negative wb_status. On error a message for
 *     the calling thread is available from wb_last_error().
 *   - Host structs passed in are copied; the caller keeps ownership.
 *   - Objects returned through an out-pointer are owned by the library and are
 *     released with the matching *_destroy call.
 *   - "stream" arguments are hipStream_t values passed as void* (NULL is the
 *     null stream). Device pointers must be device memory or pinned host memory
 *     addressable from the current HIP device, and 16-byte aligned. Calls that
 *     launch work refuse (WB_EINVAL, before anything is enqueued) null and
 *     misaligned pointers, pageable host memory and unknown addresses, and
 *     device allocations smaller than the call needs.
 *   - The library never allocates device memory. It allocates host memory and,
 *     for the pointer tables of wb_pack/wb_unpack, a small pinned host buffer;
 *     wb_unpack_round_noalloc uses a fixed device array the library's code
 *     object holds on each GPU.
 */
#ifndef WB_H
#define WB_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum wb_status {
  WB_OK = 0,
  WB_EINVAL = -1,        /* bad argument: null pointer, bad degree, out-of-range rank or index */
  WB_EUNSUPPORTED = -2,  /* valid request outside what the library implements */
  WB_ENOMEM = -3,        /* host allocation failed */
  WB_EHIP = -4,          /* a HIP runtime call failed (message has the HIP error) */
  WB_ESIZE = -5          /* caller buffer too small (see the "needed" out-argument) */
} wb_status;

typedef enum wb_dtype { WB_F32 = 0, WB_BF16 = 1, WB_F8E4M3 = 2, WB_DTYPE_NONE = -1 } wb_dtype;

/* Model families whose checkpoint catalog wb_describe_layout knows. The catalog
 * is the ordered list of checkpoint tensors, each at most 2-D ([rows, cols];
 * vectors are [1, n]):
 *   DENSE    : embed [V,H]; per layer attn_norm [1,H], q [nq*hd,H], k, v [nkv*hd,H],
 *              o [H,nq*hd], mlp_norm [1,H], gate, up [F,H], down [H,F];
 *              final_norm [1,H]; lm_head [V,H]
 *   MIXTRAL  : embed; per layer the six attention tensors, router [E,H], then for
 *              each expert e gate_e, up_e [F,H], down_e [H,F]; final_norm; lm_head
 *   MOE_ONLY : per layer router [E,H], shared gate, up [F*S,H], shared down
 *              [H,F*S], then the E routed experts as above (no attention). */
typedef enum wb_family { WB_FAMILY_DENSE = 0, WB_FAMILY_MIXTRAL = 1, WB_FAMILY_MOE_ONLY = 2 } wb_family;

typedef struct wb_model_shapes {
  int32_t family;             /* wb_family */
  int32_t num_layers;
  int32_t hidden;             /* H */
  int32_t num_heads;          /* nq */
  int32_t num_kv_heads;       /* nkv */
  int32_t head_dim;           /* hd */
  int32_t ffn;                /* F (per expert for MoE families) */
  int32_t vocab;              /* V */
  int32_t num_experts;        /* E */
  int32_t num_shared_experts; /* S */
} wb_model_shapes;

/* Layout styles:
 *   FSDP_FLAT : FSDP1-style flat units (embed; each layer, or each layer's
 *               non-expert part and each expert-parallel group's experts;
 *               final_norm + lm_head), each unit's concatenation padded to a
 *               multiple of fsdp; rank f holds the f-th equal piece as a 1-D
 *               tensor. Non-expert units are replicated over ep and dp.
 *               rank = (dp_i * ep + ep_i) * fsdp + f.
 *   MEGATRON  : trainer tensor/expert parallel. Vocab-row embed/lm_head; fused
 *               qkv grouped per kv head [q heads of the group; k; v]; fused
 *               gate_up [gate rows; up rows]; row-parallel o/down column slabs,
 *               stored transposed when transposed_row_parallel is set; MoE
 *               experts stacked per ep rank (w1, w3 [E/ep,F,H], w2), router and
 *               shared expert replicated (MoE needs tp == 1).
 *               rank = (dp_i * ep + ep_i) * tp + tp_i.
 *   SERVING   : rollout tensor/expert parallel. qkv [q slab; k slab; v slab];
 *               gate_up [gate slab; up slab]; o/down column slabs; experts
 *               stacked w13 [E/ep, 2F/tp, H] (expert j = [gate_j; up_j]) and
 *               w2 [E/ep, H, F/tp]; attention, norms, router replicated over ep.
 *               With quant_dtype = WB_F8E4M3 the linear weights (qkv, o,
 *               gate_up, down, w13, w2, shared w13/w2) are fp8 E4M3FN, each
 *               followed by an fp32 scale tensor [batch, ceil(rows/B), ceil(cols/B)].
 *               rank = (dp_i * ep + ep_i) * tp + tp_i. */
typedef enum wb_style { WB_STYLE_FSDP_FLAT = 0, WB_STYLE_MEGATRON = 1, WB_STYLE_SERVING = 2 } wb_style;

typedef struct wb_parallelism {
  int32_t style;                   /* wb_style */
  int32_t dtype;                   /* local parameter dtype: WB_F32 or WB_BF16 */
  int32_t tp, ep, fsdp, dp;        /* degrees, each >= 1 */
  int32_t transposed_row_parallel; /* MEGATRON only: 0 or 1 */
  int32_t quant_dtype;             /* SERVING only: WB_DTYPE_NONE or WB_F8E4M3 */
  int32_t quant_block;             /* block edge for quant_dtype (1..128) */
} wb_parallelism;

typedef struct wb_layout_t wb_layout_t;
typedef struct wb_plan_t wb_plan_t;
typedef struct wb_probe_t wb_probe_t;

/* One slice-copy (Sec. 3.1): rows r0..r1-1, cols c0..c1-1 of checkpoint tensor t
 * are stored in local tensor u of the rank at
 *   local[u][base + (i - r0) * ld + (j - c0)]   (transposed == 0)
 *   local[u][base + (j - c0) * ld + (i - r0)]   (transposed == 1)
 * Offsets are in elements of the local tensor's dtype. */
typedef struct wb_placement {
  int32_t t, u;
  int64_t r0, r1, c0, c1;
  int64_t base, ld;
  int32_t transposed;
  int32_t reserved;
} wb_placement;

typedef struct wb_tensor_desc {
  const char* name;
  int64_t rows, cols;
} wb_tensor_desc;

typedef struct wb_local_info {
  const char* name;      /* valid while the layout lives */
  int32_t dtype;         /* wb_dtype */
  int32_t quant_block;   /* > 0 for fp8 tensors with a scale companion */
  int64_t batch, rows, cols;
  int32_t scale_index;   /* index of the companion scale tensor, or -1 */
  int32_t scales_index;  /* for a scale tensor: index of the tensor it scales, else -1 */
} wb_local_info;

/* ---- layouts --------------------------------------------------------- */

/* All ranks of one side for a known model family and parallelism style.
 * Errors: WB_EINVAL (null, degree < 1, degrees that do not divide vocab, heads,
 * kv heads, ffn or experts, bad dtype), WB_EUNSUPPORTED (style/family
 * combinations listed above as unsupported). */
int wb_describe_layout(const wb_model_shapes* shapes, const wb_parallelism* par, wb_layout_t** out);

/* Generic layouts (a source map declared directly, e.g. recovered by probing a
 * weight loader). wb_layout_add_local with dtype WB_F8E4M3 and quant_block > 0
 * also appends the fp32 scale companion right after it. */
int wb_layout_create(const wb_tensor_desc* catalog, int32_t num_tensors, int32_t num_ranks, wb_layout_t** out);
int wb_layout_add_local(wb_layout_t* layout, int32_t rank, const char* name, int32_t dtype, int64_t batch,
                        int64_t rows, int64_t cols, int32_t quant_block, int32_t* out_index);
/* Errors: WB_EINVAL when the rectangle or the addressed local elements fall
 * outside the tensor, or when u names a scale tensor. */
int wb_layout_add_placement(wb_layout_t* layout, int32_t rank, const wb_placement* p);

int wb_layout_num_ranks(const wb_layout_t* layout, int32_t* out);
int wb_layout_num_tensors(const wb_layout_t* layout, int32_t* out);
int wb_layout_tensor(const wb_layout_t* layout, int32_t t, wb_tensor_desc* out);
int wb_layout_num_locals(const wb_layout_t* layout, int32_t rank, int32_t* out);
int wb_layout_local(const wb_layout_t* layout, int32_t rank, int32_t index, wb_local_info* out);
int wb_layout_num_placements(const wb_layout_t* layout, int32_t rank, int32_t* out);
int wb_layout_placement(const wb_layout_t* layout, int32_t rank, int32_t index, wb_placement* out);
/* Canonical text form. Writes at most cap bytes (NUL-terminated) and the full
 * size including the NUL to *needed; WB_ESIZE if cap is too small. */
int wb_layout_dump(const wb_layout_t* layout, char* buf, size_t cap, size_t* needed);
void wb_layout_destroy(wb_layout_t* layout);

/* ---- plans ----------------------------------------------------------- */

typedef enum wb_role { WB_SENDER = 0, WB_RECEIVER = 1 } wb_role;

/* Build the global routing plan of the two layouts (deterministic: every rank
 * computes the same assignment) and keep the view of one rank: a trainer rank
 * for WB_SENDER, a rollout rank for WB_RECEIVER. Canonical rules:
 *   groups  : identical trainer rectangles of a tensor form one group; distinct
 *             groups must be disjoint;
 *   order   : rollout rank ascending, its placements in layout order, groups by
 *             (r0, c0, r1, c1); each overlap is a region;
 *   split   : a region held by k > 1 ranks is cut into k near-equal parts
 *             (rows if it has >= k rows, else columns) handed out, largest
 *             first, to the owner furthest below its even share of that owner
 *             set (ties: lower part index, lower rank);
 *   wire    : per (sender, receiver) the payloads in canonical order, each a
 *             row-major copy of its rectangle in the sender dtype starting at a
 *             multiple of 256 bytes; buffers hold regions by ascending peer,
 *             each starting at a multiple of 4096 bytes.
 * A receiver's fp8 block tables are built by up to WB_PLAN_THREADS host
 * threads (environment, 1..64, for any plan with fp8 blocks; default: one for
 * fewer than 32768 blocks, else the CPUs the process may run on, at most 16);
 * the plan does not depend on the number.
 * Errors: WB_EINVAL (null, rank out of range, catalogs differ, a rollout
 * element held by no trainer, rollout tensors not exactly covered),
 * WB_EUNSUPPORTED (overlapping non-identical trainer rectangles, replicas with
 * different dtypes, an unsupported cast, an fp8 placement that is transposed
 * or not a sub-rectangle of one matrix, quant_block > 128). */
int wb_plan(const wb_layout_t* trainer, const wb_layout_t* rollout, int32_t role, int32_t rank, wb_plan_t** out);

/* The same plan cut into rounds (Sec. 3.2: the model is transferred in roughly
 * equal chunks, one per round, so that buffers stay bounded; App. D: the round
 * count follows from the registered-buffer budget). round_budget > 0 bounds the
 * bytes any sender or receiver handles in one round: checkpoint tensors are
 * grouped into units (tensors whose images share an fp8 destination block are
 * one unit, so no block spans rounds) and each round is a run of units in
 * catalog order. Filling with a cap X, a unit that would push some rank past
 * X opens the next round (so a rank goes past X only through the round's
 * first unit, one larger than X); the number of rounds n is what filling with the
 * budget needs, and the rounds are the filling with the smallest cap X <=
 * budget that still needs only n rounds, so they come out about equal.
 * Segments, owners and balance equal those of wb_plan; each round has its own
 * wire offsets under the same rules. round_budget == 0 gives one round
 * (wb_plan).
 * Errors: as wb_plan; WB_EINVAL for a negative budget. */
int wb_plan_rounds(const wb_layout_t* trainer, const wb_layout_t* rollout, int32_t role, int32_t rank,
                   int64_t round_budget, wb_plan_t** out);
int wb_plan_num_rounds(const wb_plan_t* plan, int32_t* out);
/* This rank's send (sender) or receive (receiver) buffer size in one round. */
int wb_plan_round_buffer_bytes(const wb_plan_t* plan, int32_t round, int64_t* out);
/* Region of a (sender, receiver) pair in one round, as wb_plan_region. */
int wb_plan_round_region(const wb_plan_t* plan, int32_t round, int32_t sender, int32_t receiver,
                         int64_t* send_offset, int64_t* recv_offset, int64_t* bytes);

int wb_plan_num_segments(const wb_plan_t* plan, int64_t* out);        /* global */
/* This rank's send or receive buffer size: the largest over the plan's rounds. */
int wb_plan_buffer_bytes(const wb_plan_t* plan, int64_t* out);
int wb_plan_num_peers(const wb_plan_t* plan, int32_t* out);           /* regions in this rank's round-0 buffer */
/* i-th region of this rank's round-0 buffer (ascending peer): peer rank, byte offset, bytes. */
int wb_plan_peer(const wb_plan_t* plan, int32_t i, int32_t* peer, int64_t* offset, int64_t* bytes);
/* Round-0 region of any (sender, receiver) pair: offset in the sender's buffer,
 * offset in the receiver's buffer, bytes (0 when the pair exchanges nothing). */
int wb_plan_region(const wb_plan_t* plan, int32_t sender, int32_t receiver, int64_t* send_offset,
                   int64_t* recv_offset, int64_t* bytes);
/* Buffer size of any sender (role WB_SENDER) or receiver (WB_RECEIVER), the
 * largest over the rounds. */
int wb_plan_rank_buffer_bytes(const wb_plan_t* plan, int32_t role, int32_t rank, int64_t* out);
/* Number of local tensors of this rank: the length of src_ptrs / dst_ptrs. */
int wb_plan_num_local_tensors(const wb_plan_t* plan, int32_t* out);
/* dtype (wb_dtype) and element count of src_ptrs[i] / dst_ptrs[i] (fp8
 * tensors' scale companions are entries of their own). Errors: WB_EINVAL. */
int wb_plan_local_tensor(const wb_plan_t* plan, int32_t i, int32_t* dtype, int64_t* numel);
/* Bytes of device workspace wb_plan_upload needs. */
int wb_plan_workspace_bytes(const wb_plan_t* plan, int64_t* out);
/* Algorithmic bytes one wb_pack or wb_unpack of this rank reads and writes. */
int wb_plan_traffic_bytes(const wb_plan_t* plan, int64_t* read_bytes, int64_t* write_bytes);
/* The same split by launch: launch 0 is the copy/cast kernel, launch 4 the
 * transpose-tile kernel (whole tiles of 128 source rows x 512 source columns
 * of 2-byte transposes; 0 otherwise), launch 1 the fp8 block kernel (receivers with fp8 tensors only;
 * 0 otherwise); launches 2 and 3 are the forward packings of exchange stages
 * 1 and 2 over all rounds (receivers of three-stage plans; 0 otherwise).
 * Launches 0, 1 and 4 add up to wb_plan_traffic_bytes. */
int wb_plan_kernel_traffic(const wb_plan_t* plan, int32_t launch, int64_t* read_bytes, int64_t* write_bytes);
/* Kernel work items of this rank: copy/cast tasks, fp8 blocks, fp8 pieces. */
int wb_plan_work_counts(const wb_plan_t* plan, int64_t* tasks, int64_t* blocks, int64_t* pieces);
/* 64-bit FNV-1a digest of the kernel work tables wb_plan_upload would copy
 * (work items, fp8 blocks and pieces, their per-round ranges and class splits)
 * and of the per-launch byte counts: equal digests mean the same kernel work,
 * whatever produced the plan (process, build, or number of planning threads). */
int wb_plan_work_digest(const wb_plan_t* plan, uint64_t* out);
/* Grid (workgroups in x and y) and workgroup size (threads) of one launch of
 * one round: launch 0 the copy/cast kernel of wb_pack_round / wb_unpack_round,
 * 4 its transpose-tile kernel (one workgroup per 128 x 512 tile), 1 the fp8
 * block kernel, 2 and 3 the forward packings of exchange stages 1 and 2. A copy/cast work item takes several workgroups (one per chunk of its
 * vectors), so the copy grid is a multiple of the work-item count; the fp8
 * grid has one workgroup per pair of pairable blocks (single-piece blocks and
 * blocks of full-width row bands) and one per other block. The grid is 0 x 0
 * for a launch that enqueues nothing. WB_EINVAL for a null argument, a launch
 * outside 0..4 or a round out of range. */
int wb_plan_launch_grid(const wb_plan_t* plan, int32_t launch, int32_t round, uint32_t* grid_x, uint32_t* grid_y,
                        uint32_t* threads);
/* Canonical text form of the global plan (one line per segment). */
int wb_plan_dump(const wb_plan_t* plan, char* buf, size_t cap, size_t* needed);

/* Copy this rank's work tables into caller-owned device memory (at least
 * wb_plan_workspace_bytes, 256-byte aligned), enqueued on stream. The caller
 * keeps the workspace alive and unmodified while the plan is used.
 * Errors: WB_EINVAL (null, too small, misaligned), WB_EHIP. */
int wb_plan_upload(wb_plan_t* plan, void* workspace, size_t bytes, void* stream);

/* Enqueue the packing kernel of a sender plan: src_ptrs[i] is local tensor i of
 * the rank (wb_plan_num_local_tensors entries), send_buf holds at least
 * wb_plan_buffer_bytes bytes. Writes every payload byte of the rank's regions;
 * bytes between payloads are left as they were. One kernel launch, and one
 * more when the rank has whole 128 x 512 tiles to transpose.
 * Errors (synchronous): WB_EINVAL (wrong role, not uploaded, null or misaligned
 * pointer), WB_EHIP (launch failure). Device faults surface at stream sync. */
int wb_pack(wb_plan_t* plan, const void* const* src_ptrs, void* send_buf, void* stream);

/* Enqueue the assembly of a receiver plan: recv_buf holds the regions of all
 * senders at the offsets the plan gives (wb_plan_peer / wb_plan_region); every
 * element of every local tensor (dst_ptrs, wb_plan_num_local_tensors entries,
 * scale tensors included) is written exactly once. One launch for copy/cast
 * work (two with whole transpose tiles) and one for fp8 blocks when the rank
 * has fp8 tensors.
 * Errors as for wb_pack. Calls on one plan must not overlap in time from several
 * host threads (the pointer tables are per plan; see wb_pack_round). */
int wb_unpack(wb_plan_t* plan, const void* recv_buf, void* const* dst_ptrs, void* stream);

/* One round of a multi-round plan: the same contracts as wb_pack / wb_unpack for
 * the round's work items and buffer (wb_plan_round_buffer_bytes). The send or
 * receive buffer is a launch argument, so consecutive rounds may alternate
 * between buffers (double buffering) at no cost. The local-tensor pointers
 * are read from a device table: a plan keeps the tables of its last four
 * pointer sets, so alternating sets costs no copy and no host wait; a new set
 * refills the least recently staged table, and the host waits only for that
 * table's staging copy from four sets before. Work on another stream that read
 * or wrote a table is waited for on the calling stream before the table is
 * read or rewritten (hipStreamWaitEvent), so calls on several streams may
 * share a plan when made from one host thread.
 * wb_pack / wb_unpack refuse (WB_EINVAL) plans with more than one round. */
int wb_pack_round(wb_plan_t* plan, int32_t round, const void* const* src_ptrs, void* send_buf, void* stream);
int wb_unpack_round(wb_plan_t* plan, int32_t round, const void* recv_buf, void* const* dst_ptrs, void* stream);

/* For callers that cannot allocate memory (code under stream capture, tight
 * serving loops, harnesses that forbid allocation): wb_unpack_round with no
 * caller workspace and no wb_plan_upload. The call stages the round's work
 * tables and the dst_ptrs table in a device array that the library holds on
 * each GPU it runs on until the process ends (32 MiB per GPU), then enqueues
 * the kernels of wb_unpack_round on stream; it allocates nothing. Every call
 * on a GPU shares that GPU's array and overwrites it: calls on one stream are
 * ordered, calls that overlap in time on one GPU (other streams, threads or
 * plans) race. The plan's host tables are the source of the staging copies:
 * keep the plan alive until the call's work has run.
 * Errors: WB_ESIZE (checked first) when the round's tables exceed the array
 * (plan with a smaller round budget); otherwise as wb_unpack_round, WB_EHIP. */
int wb_unpack_round_noalloc(wb_plan_t* plan, int32_t round, const void* recv_buf, void* const* dst_ptrs, void* stream);

/* ---- three-stage plans: rollout-side de-duplication and exchange ------ */

/* The plan of wb_plan_rounds plus rollout-side de-duplication and the two
 * exchange stages (Sec. 3.2: each rollout node should take in one copy of what
 * it needs over the inter-node network and share it inside the node; Figure 5).
 * node_size > 0 groups rollout ranks into nodes of node_size consecutive ranks
 * (node_size == 0 gives exactly wb_plan_rounds). Rules on top of wb_plan's:
 *   rollout groups : identical rollout rectangles of a tensor held by m > 1
 *                    ranks are cut into m parts by wb_plan's split rule and
 *                    handed out over the holders by its deficit rule counted in
 *                    elements (groups taken when their lowest holder's
 *                    placement is visited); in the receive stage (0) every
 *                    holder asks the trainers for its parts only;
 *   external (1)   : every stage-0 segment of such a group is forwarded, byte
 *                    for byte, to one holder in each other node: position
 *                    (i mod n_v) of that node's holder list, where i is the
 *                    position of the forwarding rank in its own node's list;
 *   internal (2)   : every stage-0 and stage-1 segment of such a group is
 *                    forwarded to each other holder in the receiver's node.
 * Forwarded payloads keep the trainer dtype. A rollout rank's receive buffer
 * holds the stage-0 regions, then the stage-1 regions, then the stage-2
 * regions, each non-empty section starting at a multiple of 4096 bytes; every
 * forwarding rank has one forward buffer per exchange stage, laid out like a
 * send buffer. wb_plan_round_buffer_bytes of a receiver covers all sections;
 * wb_unpack_round reads all of them, so it runs after both exchange stages of
 * the round have landed.
 * Errors: as wb_plan_rounds; WB_EINVAL for a negative node size or a rollout
 * rank holding one rectangle twice. */
int wb_plan_exchange(const wb_layout_t* trainer, const wb_layout_t* rollout, int32_t role, int32_t rank,
                     int64_t round_budget, int32_t node_size, wb_plan_t** out);
int wb_plan_node_size(const wb_plan_t* plan, int32_t* out);
/* Region of a (sender, receiver) pair in one stage of one round: stage 0 as
 * wb_plan_round_region; stages 1 and 2 pair rollout ranks, send_offset in the
 * sender's forward buffer of that stage, recv_offset in the receiver's whole
 * receive buffer. bytes is 0 when the pair exchanges nothing. */
int wb_plan_stage_region(const wb_plan_t* plan, int32_t round, int32_t stage, int32_t sender, int32_t receiver,
                         int64_t* send_offset, int64_t* recv_offset, int64_t* bytes);
/* This receiver's forward buffer size for exchange stage 1 or 2 in one round
 * (round -1: the largest over the rounds); 0 for senders. */
int wb_plan_forward_bytes(const wb_plan_t* plan, int32_t round, int32_t stage, int64_t* out);

/* One segment of the global plan (0 <= i < wb_plan_num_segments), in the order
 * of wb_plan_dump: sender and receiver ranks (a trainer and a rollout rank in
 * stage 0, rollout ranks in stages 1 and 2), checkpoint tensor and rectangle,
 * stage and round, the trainer placement (stage 0; -1 otherwise) and the
 * receiver's placement, offsets in the sender's send or forward buffer and in
 * the receiver's receive buffer, for forwarded segments the offset of the
 * forwarded bytes in the sender's receive buffer (else 0) and the index of the
 * stage-0 segment they left the trainers in (a stage-0 segment's own index),
 * and the payload bytes. Errors: WB_EINVAL (null, index out of range). */
typedef struct wb_segment_info {
  int32_t sender, receiver, tensor, stage, round, src_placement, dst_placement, reserved;
  int64_t r0, r1, c0, c1;
  int64_t send_offset, recv_offset, src_offset, origin, bytes;
} wb_segment_info;
int wb_plan_segment(const wb_plan_t* plan, int64_t i, wb_segment_info* out);
/* Enqueue the forward packing of a receiver plan for exchange stage 1 or 2 of
 * one round: every payload this rank forwards in that stage is copied from
 * where it landed in recv_buf (wb_plan_round_buffer_bytes) to its offset in
 * fwd_buf (wb_plan_forward_bytes). One launch of the copy kernel; nothing is
 * enqueued (and the buffers are not checked) when the rank forwards nothing.
 * Stage 1 reads the stage-0 section, stage 2 the stage-0 and stage-1 sections,
 * so each must have landed. Errors as for wb_pack; wb_plan_kernel_traffic
 * launches 2 and 3 give its algorithmic bytes. */
int wb_forward_round(wb_plan_t* plan, int32_t round, int32_t stage, const void* recv_buf, void* fwd_buf,
                     void* stream);

void wb_plan_destroy(wb_plan_t* plan);

/* ---- source-map probing (Sec. 3.1; App. B, Algorithm 1) ---------------- */

/* Layouts can also be discovered from a weight loader that copies values
 * unchanged (a black box), instead of being declared. Every checkpoint element
 * gets the identifier 2^24 + its flat position in the checkpoint (catalog
 * order, row-major; 0 marks an element no loader wrote). The checkpoint is
 * loaded once per 16-bit chunk of the identifiers (wb_probe_chunks passes);
 * after pass k the caller runs wb_diff2_carry over the loaded local tensors
 * (or wb_diff2 on each) and hands the entries to wb_probe_record. The library
 * sums 2^(16 k) times pass k's entries, which is exactly diff2 of the full
 * identifier field because diff2 is linear and the carries telescope, and
 * wb_probe_scan turns the result into slice-copy placements without building
 * the identifier field: between rows and columns that hold entries the field
 * is a bilinear polynomial given by prefix sums of four moments of the
 * entries; it must be affine inside every such cell, cells are merged into
 * maximal affine rectangles, and each rectangle is decoded (flat runs as a
 * partial head row, whole rows and a partial tail row; slabs; transposed
 * slabs; anything else row by row or element by element).
 * ckpt_dtype is WB_F32 or WB_BF16: the chunk travels as the bit pattern of a
 * bf16 element or as the exact value of an f32 element.
 * Errors: WB_EINVAL (null, bad catalog), WB_EUNSUPPORTED (other dtypes). */
int wb_probe_create(const wb_tensor_desc* catalog, int32_t num_tensors, int32_t ckpt_dtype, wb_probe_t** out);
/* Number of loading passes and identifier bits per pass (16). */
int wb_probe_chunks(const wb_probe_t* probe, int32_t* num_chunks, int32_t* chunk_bits);
/* Identifier of element (0, 0) of checkpoint tensor t. */
int wb_probe_first_id(const wb_probe_t* probe, int32_t t, int64_t* id);
/* Declare a local tensor of the probed rank, seen as a [batch * rows, cols]
 * field; dtype is the checkpoint dtype (value-preserving loaders only). */
int wb_probe_add_local(wb_probe_t* probe, const char* name, int32_t dtype, int64_t batch, int64_t rows, int64_t cols,
                       int32_t* index);
/* Host arrays of n entries of pass `chunk` for local tensor `local`: flat
 * element index and value (as wb_diff2 or wb_diff2_carry write them, widened
 * to int64), added times 2^(16 chunk). Entries of wb_diff2_batch over all
 * passes at once are recorded as chunk 0. Errors: WB_EINVAL (index or chunk out of range). */
int wb_probe_record(wb_probe_t* probe, int32_t local, int32_t chunk, const int64_t* index, const int64_t* value,
                    int64_t n);
/* Fill rank `rank` of `layout` (made by wb_layout_create over the same catalog,
 * with no local tensors yet) with the probe's local tensors and the placements
 * recovered from the recorded passes. Errors: WB_EINVAL (catalogs differ, rank
 * already filled), WB_EUNSUPPORTED (a field that is not made of slice copies
 * of identifiers: the loader changed values or mixed elements). */
int wb_probe_scan(const wb_probe_t* probe, wb_layout_t* layout, int32_t rank);
void wb_probe_destroy(wb_probe_t* probe);

/* Write chunk `chunk` (16 bits, chunk_bits = 16) of the identifiers
 * first_id .. first_id + numel - 1 into a checkpoint tensor of dtype WB_BF16
 * (bit pattern) or WB_F32 (exact value): Algorithm 1, MakeIdChunk. One launch.
 * dst needs only element alignment. Errors: WB_EINVAL (null, misaligned, bad
 * dtype or chunk). */
int wb_make_ids(void* dst, int32_t dtype, int64_t numel, int64_t first_id, int32_t chunk, int32_t chunk_bits,
                void* stream);
/* diff2 (Eqs. diff1, diff2: the outer product of [1, -2, 1] with itself, the
 * field taken as 0 above and left of the tensor) of the chunk field held by a
 * loaded local tensor src of dtype WB_BF16 or WB_F32 seen as [rows, cols];
 * appends the non-zero entries to the device arrays index (flat position) and
 * value (at most `capacity` of them, order unspecified) and sets the device
 * counter *count to the number of non-zero entries (which may exceed
 * capacity: then call again with more room). The counter is reset by the
 * call. One small and one stencil launch; the stencil reads each element about
 * once. src, index and value need only element alignment. Errors: WB_EINVAL
 * (null, misaligned, bad dtype or shape). */
int wb_diff2(const void* src, int32_t dtype, int64_t rows, int64_t cols, int64_t* index, int32_t* value,
             int64_t capacity, uint64_t* count, void* stream);
/* A field for wb_diff2_batch: `passes` (1 to 3) device arrays data[0..passes)
 * of dtype WB_BF16 or WB_F32, each seen as [rows, cols] (row-major,
 * contiguous, element-aligned). Its value at (i, j) is the sum over k of
 * 2^(16 k) times the chunk held by data[k] (bf16 bit pattern or exact f32
 * value): with data[k] the loaded tensor after probing pass k, that is the
 * identifier field itself. rows or cols may be 0 (a field with no entries). */
typedef struct wb_field {
  const void* data[3];
  int32_t dtype;
  int32_t passes;
  int64_t rows, cols;
} wb_field;
/* Device workspace bytes wb_diff2_batch needs for these n fields (its
 * tables: 56 bytes per field, then 24 per workgroup of the launch; 0 when no
 * field has elements). Errors: WB_EINVAL (bad field). */
int wb_diff2_batch_workspace(const wb_field* fields, int32_t n, size_t* bytes);
/* diff2 of n fields in one stencil launch (Algorithm 1 runs diff2 over every
 * loaded tensor after each pass). Because diff2 is linear, a field of several
 * passes gives the sum over k of 2^(16 k) times diff2 of pass k, formed before
 * the stencil: the entries that chunk wrap-arounds leave in single passes
 * cancel inside the launch, and only the identifier field's own entries (at
 * most 16 per slice copy) come out. Values are int64 (identifiers below 2^48).
 * An entry's index is its flat position in the concatenation of the fields in
 * order: field f's element (i, j) is the sum over g < f of rows_g * cols_g,
 * plus i * cols_f + j. index, value (8-byte aligned), capacity and count as
 * for wb_diff2 (count is the total over all fields). workspace is device
 * memory of at least wb_diff2_batch_workspace bytes, 8-byte aligned, owned by
 * the caller; the call copies the tile table into it on `stream` and waits
 * for that copy (so it returns after the stream's earlier work), and the
 * workspace must stay untouched until the launch has run. Errors: WB_EINVAL
 * (null, misaligned, bad field, workspace too small, more than 2^31 - 1
 * tiles), WB_EHIP. */
int wb_diff2_batch(const wb_field* fields, int32_t n, void* workspace, size_t workspace_bytes, int64_t* index,
                   int64_t* value, int64_t capacity, uint64_t* count, void* stream);

/* Device workspace bytes wb_diff2_carry needs for these n one-pass fields
 * and room for carry_capacity carries per pass: the tile tables, 2 KiB of
 * counters, two carry tables of 16-byte slots, each as many slots as the
 * smallest power of two at least twice carry_capacity (and 64), and 1028
 * bytes per stencil workgroup for staging its carries. Errors:
 * WB_EINVAL (bad field, a field of more than one pass, carry_capacity outside
 * 1..2^36). */
int wb_diff2_carry_workspace(const wb_field* fields, int32_t n, int64_t carry_capacity, size_t* bytes);
/* One probing pass with carries (App. B, Algorithm 1: ExpandCarry and
 * EmitCarry), for loading passes that are not kept: fields are the loaded
 * local tensors after pass `pass` (one pass each, the same fields in the same
 * order every pass), `last` is non-zero for the final pass. With D = diff2 of
 * the pass's chunk field and Q the carries pass - 1 left (none for pass 0),
 * S = D + Q; a pass other than the last appends (position, S mod 2^16) where
 * that is non-zero and keeps floor(S / 2^16) as its carries, the last appends
 * S whole. Then the sum over passes of 2^(16 pass) times the appended values
 * is diff2 of the identifier field, every value of a pass but the last lies
 * in 1..65535, and entries appear only where diff2 of the identifier field is
 * non-zero (next to slice-copy corners): a chunk's wrap-arounds stay in the
 * carries, on the device. Positions, index, value, capacity and count are as
 * for wb_diff2_batch (the counter is reset by the call). *carries (device,
 * 8-byte aligned) gets the number of carries the pass kept (0 for the last
 * pass); above carry_capacity (or, very rarely, when a carry found no free
 * slot near its hash, reported as carry_capacity + 1) carries may be lost and
 * this and later passes are wrong: start again from pass 0 with more room. A pass
 * whose count exceeded capacity can be run again with more room (same
 * workspace, same fields). workspace: device memory of at least
 * wb_diff2_carry_workspace bytes, 8-byte aligned, owned by the caller, the
 * same buffer with the same carry_capacity for every pass of one probe (it
 * holds the carries between passes). The call copies the tile table into it
 * on `stream` and waits for that copy. Passes on one workspace must not
 * overlap. Six launches at most; the stencil reads each element about once.
 * Errors: as for wb_diff2_batch, and WB_EINVAL for a field of more than one
 * pass, a negative pass, a null or misaligned carries, carry_capacity outside
 * 1..2^36. */
int wb_diff2_carry(const wb_field* fields, int32_t n, int32_t pass, int32_t last, int64_t carry_capacity,
                   void* workspace, size_t workspace_bytes, int64_t* index, int64_t* value, int64_t capacity,
                   uint64_t* count, uint64_t* carries, void* stream);

/* Message of the calling thread's last failed call ("" if none). */
const char* wb_last_error(void);
const char* wb_version(void);

#ifdef __cplusplus
}
#endif

#endif /* WB_H */
