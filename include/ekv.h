/*
 * ekv.h -- C ABI of libekv, the MI355X (gfx950) mixed-fidelity paged KV
 * attention library.
 *
 * Method: ElasticKV ("Does Execution Require Target KV Fidelity? A
 * Mixed-Fidelity KV Runtime for LLM Serving").  Every KV element exists in
 * one of two executable states:
 *
 *   TARGET -- the native 16-bit word (bf16 or fp16);
 *   BASE   -- the high-order byte of that word, executed with a zero low
 *             byte; the low byte (the refinement bits) restores TARGET
 *             exactly (paper §3, opening paragraph; App. B.2, App. B.3).
 *
 * Memory layout (all in device memory, all owned by the caller):
 *
 *   pool        uint16 [num_blocks][2][num_kv_heads][page_size][head_dim]
 *               plane 0 = K, plane 1 = V.  A physical block holds
 *               page_size tokens of every KV head (paged KV, §2.1).
 *   block_table int32  [batch][max_blocks]: logical block i of sequence s
 *               lives in physical block block_table[s][i].
 *   tags        uint8  [batch][max_blocks]: 0 = TARGET, 1 = BASE; equal
 *               for the two members of a pair.
 *
 * Pairs (§3.1): logical blocks (2j, 2j+1) of one sequence.  A BASE pair is
 * packed into ONE physical block -- the block that held member 0 -- and both
 * block-table entries point at it.  Inside it, each plane's bytes are
 * uint8 [num_kv_heads][member][page_size][head_dim], so for every
 * (plane, head) the 4 KiB that a TARGET block uses for that head hold
 * [BASE bytes of member 0 | BASE bytes of member 1].  TARGET pairs keep the
 * native layout.  Only pairs of two full blocks can be BASE.
 *
 * Refinement bytes of one pair ("lo" buffers) are exactly one block's
 * worth: uint8 [2][num_kv_heads][member][page_size][head_dim].
 *
 * Conventions shared by every call:
 *   - Every call that takes a hipStream_t is asynchronous on that stream and
 *     never synchronises; errors detected on the host are returned before
 *     anything is enqueued; a launch failure returns EKV_ERR_HIP.
 *   - The library allocates no device memory.  Scratch space is passed in
 *     by the caller (see ekv_decode_workspace_bytes), or is a static array
 *     inside the library (ekv_attn_decode_noalloc; the EKV_DEBUG report).
 *     The EKV_DEBUG=1 mode (below) synchronises.
 *   - Host-side checks cover shapes and pointers.  Checks that need the
 *     contents of device arrays (a tag that differs inside a pair, an
 *     already-BASE pair in a demotion list) are done by the ekv_check_*
 *     functions on host mirrors, or on the device by the ekv_validate_*
 *     functions; the other device calls assume valid lists.
 *     Still, no device-side value makes a call touch memory outside the
 *     arrays it was given: block-table entries and lengths are clamped into
 *     the pool and the table, prefill query offsets into [0, total_q], and
 *     append slots and transition-list entries that point outside the pool
 *     or the table are skipped (a skipped demotion reports freed_out[i] =
 *     -1).  Results for invalid lists are otherwise undefined.
 *   - Supported: head_dim 128, page_size 16, dtype bf16, fp16 or e5m2 (the
 *     8-bit pools below), num_q_heads / num_kv_heads in {1, 2, 4, 8, 16}.  Other shapes return
 *     EKV_ERR_UNSUPPORTED.
 *   - No C++ exception crosses this interface: a host-side failure inside
 *     the library (host memory exhausted) returns EKV_ERR_HOST, with nothing
 *     enqueued.
 *   - ekv_last_error() returns a text describing the last failure on the
 *     calling thread.
 */
#ifndef EKV_H
#define EKV_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t ekv_status;
enum {
  EKV_OK = 0,
  EKV_ERR_INVALID = 1,      /* bad argument or transition list */
  EKV_ERR_UNSUPPORTED = 2,  /* valid but not implemented for this shape */
  EKV_ERR_HIP = 3,          /* a HIP runtime call failed */
  EKV_ERR_HOST = 4          /* a host-side failure inside the library (out of host memory); nothing was enqueued */
};

enum { EKV_DTYPE_BF16 = 0, EKV_DTYPE_FP16 = 1, EKV_DTYPE_FP32 = 2, EKV_DTYPE_E5M2 = 3 };

/*
 * 8-bit TARGET / 4-bit BASE pools (the paper notes the contract carries
 * over to an 8-bit TARGET with a 4-bit executable state, App. C.5):
 * dtype EKV_DTYPE_E5M2 stores TARGET as FP8 E5M2 bytes -- the high byte of
 * an FP16 word, executed as that FP16 word with a zero low byte -- in
 *   pool  uint8 [num_blocks][2][num_kv_heads][page_size][head_dim].
 * BASE is the byte's high nibble (sign and top three exponent bits),
 * executed with a zero low nibble; the low nibble refines it exactly.  A
 * BASE pair packs both members' nibbles into member 0's block: per
 * (plane, head), the 2 KiB of a TARGET tile hold [member 0 | member 1],
 * each uint8 [page_size][head_dim / 2] with element e of a row in byte
 * e / 2, low nibble for even e.  Refinement nibbles ("lo") of a pair use the
 * same layout and fill exactly one 8-bit block.  Queries are FP16 and
 * outputs FP16 or FP32.  Every entry point accepts such a pool: decode,
 * prefill, append, demote and refine (also multi-layer and staged).
 */

/* Batch execution mode (§3.2; App. B.3): NATIVE for TARGET-only batches;
 * STRUCTURED when every sequence is TARGET* BASE* TARGET* (described by its
 * boundaries); GENERAL when some sequence needs the explicit tag table. */
enum { EKV_MODE_NATIVE = 0, EKV_MODE_STRUCTURED = 1, EKV_MODE_GENERAL = 2 };

enum { EKV_TAG_TARGET = 0, EKV_TAG_BASE = 1 };

typedef struct {
  void* kv;               /* device pool, layout above */
  int32_t num_blocks;
  int32_t num_kv_heads;
  int32_t page_size;      /* 16 */
  int32_t head_dim;       /* 128 */
  int32_t dtype;          /* EKV_DTYPE_BF16, EKV_DTYPE_FP16 or EKV_DTYPE_E5M2 */
} ekv_pool;

typedef struct {
  int32_t batch;
  int32_t num_q_heads;
  int32_t max_blocks;          /* row length of block_table and tags */
  int32_t mode;                /* EKV_MODE_*, as returned by ekv_lower */
  int32_t max_seq_len;         /* upper bound on seq_lens[] (0: max_blocks*page_size) */
  const int32_t* seq_lens;     /* device int32 [batch] */
  const int32_t* block_table;  /* device int32 [batch][max_blocks] */
  const uint8_t* tags;         /* device uint8 [batch][max_blocks]; may be NULL in NATIVE mode */
  const int32_t* boundaries;   /* device int32 [batch][2] or NULL (NULL: tags for every sequence) */
} ekv_batch;

/* Text for a status code (static storage). */
const char* ekv_status_string(ekv_status s);

/* Message for the last failing call on this thread (static thread-local storage). */
const char* ekv_last_error(void);

/* Library version as "major.minor.patch". */
const char* ekv_version(void);

/*
 * Dispatch metadata lowering (§3.2; App. B.3), host only.
 * h_tags [batch][max_blocks], h_seq_lens [batch]: host mirrors.
 * Writes *mode_out (EKV_MODE_*) and h_boundaries_out [batch][2]: for a
 * sequence whose visible pair modes read TARGET* BASE* TARGET*, the pair
 * range [b0, b1) that is BASE (b0 == b1 when none); (-1, -1) for any other
 * sequence.  Only the ceil(len/page_size) blocks holding tokens are read.
 * Errors: EKV_ERR_INVALID on NULL pointers, negative sizes, a length beyond
 * max_blocks*page_size, or a pair whose two tags differ.
 */
ekv_status ekv_lower(const uint8_t* h_tags, const int32_t* h_seq_lens, int32_t batch,
                     int32_t max_blocks, int32_t page_size, int32_t* mode_out,
                     int32_t* h_boundaries_out);

/*
 * Bytes of device scratch that ekv_attn_decode needs for this pool and
 * batch: merge counters and the split-KV partial results of the (sequence,
 * KV head)s that a launch cuts, two slots of G = num_q_heads / num_kv_heads
 * partial rows per workgroup of the persistent grid.  The size depends on
 * the group size and on the batch's work (number of sequences times its
 * length bound) only up to the grid's cap of 4096 workgroups, not on the
 * mode, the lengths themselves or the device: a workspace of this size
 * serves every call whose batch needs no more, on any device.  At most
 * 2 * 4096 * G * 520 + 32 KiB bytes.  Returns 0 for unsupported shapes.
 */
size_t ekv_decode_workspace_bytes(const ekv_pool* pool, const ekv_batch* batch);

/*
 * Prepare a decode workspace for first use: fills ws_bytes bytes of ws
 * with zeros on the stream (a kernel, not a memset).  The merge counters
 * must read zero when a decode starts; every decode call leaves them at
 * zero (they keep one place whatever the batch, so calls with different
 * batches may share a workspace), so this is needed once after allocation
 * (or after ws was used for anything else).  A zero-filled allocation
 * needs no call.
 * Errors: EKV_ERR_INVALID (NULL ws with nonzero size, size not a multiple
 * of 4), EKV_ERR_HIP.
 */
ekv_status ekv_decode_workspace_init(void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * Decode attention, one query token per sequence (§3.2; App. B.3): for
 * sequence s and query head h (KV head h / (Hq/Hkv)),
 *   out[s][h] = softmax(scale * q[s][h] . K_s^T) V_s
 * over the seq_lens[s] cached tokens, each KV block read in its mode: TARGET
 * words as they are, BASE bytes placed in the high byte with a zero low
 * byte.  batch->mode selects the native path (no tag is read) or the
 * elastic path; in the elastic path a sequence with boundaries[s][0] >= 0
 * uses its boundaries and any other sequence reads its tags.
 *   q    device [batch][num_q_heads][head_dim], pool dtype
 *   out  device [batch][num_q_heads][head_dim], out_dtype = pool dtype or EKV_DTYPE_FP32
 *   ws   device scratch of at least ekv_decode_workspace_bytes() bytes,
 *        16-byte aligned, prepared by ekv_decode_workspace_init (or
 *        zero-filled) before its first use; calls sharing one ws must be
 *        ordered on one stream
 * A sequence of length 0 yields zeros.
 * Errors: EKV_ERR_INVALID (NULL pointers, sizes, workspace too small or
 * misaligned, NATIVE mode expected but tags needed), EKV_ERR_UNSUPPORTED,
 * EKV_ERR_HIP.
 */
ekv_status ekv_attn_decode(const ekv_pool* pool, const ekv_batch* batch, const void* q,
                           void* out, int32_t out_dtype, float scale, void* ws, size_t ws_bytes,
                           hipStream_t stream);

/*
 * Append, then decode, in one launch (§3.2: a decoded token's new K/V
 * enter in TARGET form, and the step's attention reads them).  The same
 * result, output and pool, as ekv_append_kv of each sequence's newest token
 * followed by ekv_attn_decode: for every s with seq_lens[s] >= 1, the token
 * at position p = seq_lens[s] - 1 takes k_new[s] / v_new[s], written to
 * block block_table[s][p / page_size], offset p % page_size, and the
 * attention over seq_lens[s] tokens reads these rows.  (seq_lens counts the
 * new token.)  The block of p must be TARGET, as for ekv_append_kv; a
 * sequence whose block of p is BASE is neither written nor patched (its
 * decode reads the pool as it is).
 *   k_new, v_new  device [batch][num_kv_heads][head_dim], pool dtype (bytes
 *                 for an 8-bit pool); read only
 * Other arguments as ekv_attn_decode; the pool is written.
 * Errors: as ekv_attn_decode (also EKV_ERR_INVALID for NULL k_new / v_new).
 */
ekv_status ekv_attn_decode_append(const ekv_pool* pool, const ekv_batch* batch, const void* q,
                                  const void* k_new, const void* v_new, void* out, int32_t out_dtype,
                                  float scale, void* ws, size_t ws_bytes, hipStream_t stream);

/*
 * ekv_attn_decode without a caller workspace and without any allocation,
 * for callers that cannot allocate device memory: code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation.  The
 * split-KV scratch is a static device array of 32 MiB inside the library
 * (one per device, held until the process ends); its device address is
 * looked up once per device on the first call there.  Each call first
 * zeroes the scratch's merge counters with a fill kernel on the stream,
 * then runs the same decode kernel as ekv_attn_decode (same results).  The
 * call allocates nothing and never synchronises; the EKV_DEBUG checks are
 * not run.  All calls on one device share the scratch: calls that may
 * overlap on one device (other streams, other threads) race and must be
 * ordered by the caller.  A batch whose launch needs more than 32 MiB of
 * scratch (2 slots of G partial rows per workgroup, plus 32 KiB) returns
 * EKV_ERR_UNSUPPORTED.  Other arguments and errors as ekv_attn_decode.
 */
ekv_status ekv_attn_decode_noalloc(const ekv_pool* pool, const ekv_batch* batch, const void* q, void* out,
                                   int32_t out_dtype, float scale, hipStream_t stream);

/*
 * Chunked-prefill attention (§3.2; App. A): sequence s contributes the new
 * rows q[cu_q[s] .. cu_q[s+1]) whose K/V have already been appended; row i
 * of the chunk sees keys 0 .. seq_lens[s] - n_s + i (causal, inclusive),
 * where n_s = cu_q[s+1] - cu_q[s] and seq_lens[s] counts the whole context.
 * The prefix may mix TARGET and BASE blocks; the chunk's blocks are TARGET.
 *   q    device [total_q][num_q_heads][head_dim], pool dtype (FP16 for an 8-bit pool)
 *   cu_q device int32 [batch+1], nondecreasing, cu_q[0] = 0, cu_q[batch] = total_q
 *   out  device [total_q][num_q_heads][head_dim], out_dtype = the query dtype or EKV_DTYPE_FP32
 *   max_q_len  upper bound on every n_s (sizes the launch)
 * Errors: as ekv_attn_decode.
 */
ekv_status ekv_attn_prefill(const ekv_pool* pool, const ekv_batch* batch, const void* q,
                            const int32_t* cu_q, int32_t total_q, int32_t max_q_len, void* out,
                            int32_t out_dtype, float scale, hipStream_t stream);

/*
 * Append new K/V rows as TARGET (§3.2: new KV is written in TARGET form).
 * Row i goes to token slot slots[i] = physical_block * page_size + offset.
 *   slots device int32 [n]; k, v device [n][num_kv_heads][head_dim], pool dtype.
 * Slots must be distinct and lie in TARGET blocks.
 * Errors: EKV_ERR_INVALID, EKV_ERR_UNSUPPORTED, EKV_ERR_HIP.
 */
ekv_status ekv_append_kv(const ekv_pool* pool, const int32_t* slots, const void* k,
                         const void* v, int32_t n, hipStream_t stream);

/*
 * Demotion TARGET -> BASE (§3.1; §3.4 "Transition protocols"; App. B.2).
 * For each listed pair i = (s, j) (device int32 pairs[n][2]), with
 * b0 = block_table[s][2j] and b1 = block_table[s][2j+1]: the high bytes of
 * both blocks are packed into b0 in place; if lo_out is not NULL the low
 * bytes go to lo_out[i] (uint8 [n][one block's bytes], device memory of the
 * current device or pinned host memory mapped for it; both ends of the
 * range are looked up before anything is enqueued, a pinned host address is
 * replaced by its device address, and any other memory -- pageable host
 * memory, another device's memory, memory the runtime cannot describe --
 * is EKV_ERR_INVALID with nothing enqueued); then
 * block_table[s][2j+1] = b0, both tags = BASE and freed_out[i] = b1 (device
 * int32 [n]).  b1's bytes are not touched.  The caller returns freed_out[]
 * to its free pool only after the stream has passed this call.
 * Errors: EKV_ERR_INVALID, EKV_ERR_UNSUPPORTED, EKV_ERR_HIP, EKV_ERR_HOST.
 */
ekv_status ekv_demote(const ekv_pool* pool, int32_t n, const int32_t* pairs,
                      int32_t* block_table, uint8_t* tags, int32_t batch, int32_t max_blocks,
                      int32_t* freed_out, uint8_t* lo_out, hipStream_t stream);

/*
 * Refinement BASE -> TARGET (§3.1; §3.3; App. B.2).  For each listed pair
 * i = (s, j) with packed block P = block_table[s][2j] and the reacquired
 * block Q = new_blocks[i] (device int32 [n]): member 0 is restored in place
 * into P and member 1 into Q from the high bytes in P and the refinement
 * bytes lo_in[i] (uint8 [n][one block's bytes], device memory or pinned
 * host memory mapped for the device, read over the host link; handled as
 * lo_out of ekv_demote); then block_table[s][2j+1] = Q and
 * both tags = TARGET.  No attention call may read these pairs concurrently
 * on another stream.
 * Errors: EKV_ERR_INVALID, EKV_ERR_UNSUPPORTED, EKV_ERR_HIP.
 */
ekv_status ekv_refine(const ekv_pool* pool, int32_t n, const int32_t* pairs,
                      const int32_t* new_blocks, int32_t* block_table, uint8_t* tags,
                      int32_t batch, int32_t max_blocks, const uint8_t* lo_in, hipStream_t stream);

/*
 * Refinement from staged bytes, the last step of asynchronous promotion
 * (App. B.2: reserve the extra block, restore from the CPU backing while the
 * BASE mapping stays executable, publish after TARGET is materialised).
 * The caller has copied pair i's refinement bytes (one block's worth, the
 * lo layout of ekv_demote) into its reserved block Q = new_blocks[i] --
 * typically a host-to-device copy from pinned memory on a copy stream --
 * and orders this call after that copy.  Then, as ekv_refine: member 0 is
 * rebuilt in place in P = block_table[s][2j], member 1 in place in Q over
 * the staged bytes, block_table[s][2j+1] = Q and both tags = TARGET.
 * Until this call the pair is BASE and its mapping untouched, so attention
 * may run on it while the copy is in flight.
 * Errors: EKV_ERR_INVALID, EKV_ERR_UNSUPPORTED, EKV_ERR_HIP.
 */
ekv_status ekv_refine_staged(const ekv_pool* pool, int32_t n, const int32_t* pairs, const int32_t* new_blocks,
                             int32_t* block_table, uint8_t* tags, int32_t batch, int32_t max_blocks,
                             hipStream_t stream);

/*
 * Staging copy of asynchronous promotion (App. B.2: the restore from the CPU
 * backing runs while the BASE mapping stays executable).  For i < n, copies
 * one block's bytes (2 * num_kv_heads * page_size * head_dim elements of the
 * pool's dtype) from h_src[i] into pool block h_new_blocks[i], the block
 * reserved for pair i, ready for ekv_refine_staged.
 *   h_src         host array [n] of addresses; each range must be memory the
 *                 current device can read: its own device memory, or pinned
 *                 host memory mapped for it (hipHostMalloc; read over the
 *                 host link by the copy kernel, without a DMA copy per block).
 *                 Both ends of every range are looked up before anything is
 *                 enqueued; an address the runtime does not know (pageable
 *                 host memory) is EKV_ERR_INVALID.
 *   h_new_blocks  host int32 [n]: distinct blocks in [0, num_blocks).
 * The sources are caller-owned and must stay valid and unchanged until the
 * stream has passed this call; the destination blocks must not be read or
 * written by other work meanwhile.  No table or tag is touched.
 * Errors: EKV_ERR_INVALID, EKV_ERR_UNSUPPORTED, EKV_ERR_HIP.
 */
ekv_status ekv_stage_blocks(const ekv_pool* pool, int32_t n, const void* const* h_src,
                            const int32_t* h_new_blocks, hipStream_t stream);

/*
 * Asynchronous promotion as one protocol (App. B.2: reserve the extra
 * block, restore it from the CPU backing while the BASE mapping stays
 * executable, publish only after TARGET is materialised), for callers that
 * drive it from C.  The caller keeps the allocator: it picks the reserved
 * blocks, owns the pinned backing and decides when to publish.
 *
 * ekv_promote_begin: ekv_stage_blocks(pool, n, h_src, h_new_blocks) on
 * copy_stream, then records `copied` on copy_stream after the copy.
 * Attention may keep running on the pairs (still BASE, mapping untouched)
 * on other streams meanwhile; hipEventQuery(copied) tells the caller when
 * publishing will not wait.
 *   copied  a hipEvent_t created by the caller (required); re-recorded here.
 * Arguments and errors otherwise as ekv_stage_blocks; nothing is enqueued
 * or recorded when the arguments are refused.
 *
 * ekv_promote_publish: makes `stream` wait for `copied` (a device-side
 * wait: the host does not block), then ekv_refine_staged on `stream` --
 * member 0 rebuilt in place, member 1 rebuilt in the reserved block over the
 * staged bytes, the table entry and both tags switched to TARGET.  So the
 * mapping is published only after the bytes it points at have landed,
 * whatever the host does in between.  Arguments and errors as
 * ekv_refine_staged (new_blocks: the device copy of h_new_blocks); the
 * arguments are checked before the wait is enqueued.
 */
ekv_status ekv_promote_begin(const ekv_pool* pool, int32_t n, const void* const* h_src,
                             const int32_t* h_new_blocks, hipEvent_t copied, hipStream_t copy_stream);
ekv_status ekv_promote_publish(const ekv_pool* pool, int32_t n, const int32_t* pairs, const int32_t* new_blocks,
                               int32_t* block_table, uint8_t* tags, int32_t batch, int32_t max_blocks,
                               hipEvent_t copied, hipStream_t stream);

/*
 * Multi-layer transitions: the same pairs demoted (or refined) in every
 * layer's pool of a model in one launch.  In paged serving every layer has
 * its own pool and all layers share one block table, so a pair is one
 * decision for all layers; the paper's synchronous demotion of one such
 * batch costs 25.44 ms per invocation (App. C.6), while its traffic is
 * 4 block-equivalents per pair per layer.  Per layer l the data change is
 * exactly that of ekv_demote / ekv_refine on pool layer_kv[l]; the block
 * table, tags and freed list are updated once, after every layer's data.
 *   pool      shape and dtype shared by every layer (pool->kv must be non-NULL
 *             -- e.g. layer 0's pool -- but is not read)
 *   layer_kv  device uint64 [num_layers]: the address of each layer's pool
 *   lo_out / lo_in  device (or mapped pinned host) uint8
 *             [n][num_layers][one block's bytes]: a pair's refinement bytes of
 *             all layers are contiguous
 * 1 <= num_layers <= 65535.  Other arguments and errors as ekv_demote /
 * ekv_refine.
 */
ekv_status ekv_demote_layers(const ekv_pool* pool, const uint64_t* layer_kv, int32_t num_layers, int32_t n,
                             const int32_t* pairs, int32_t* block_table, uint8_t* tags, int32_t batch,
                             int32_t max_blocks, int32_t* freed_out, uint8_t* lo_out, hipStream_t stream);
ekv_status ekv_refine_layers(const ekv_pool* pool, const uint64_t* layer_kv, int32_t num_layers, int32_t n,
                             const int32_t* pairs, const int32_t* new_blocks, int32_t* block_table,
                             uint8_t* tags, int32_t batch, int32_t max_blocks, const uint8_t* lo_in,
                             hipStream_t stream);

/*
 * Host-side validation of a transition list against host mirrors (App. B.1:
 * only demotable TARGET pairs and promotable BASE pairs are offered).
 * kind 0 = demotion (pairs must be TARGET), 1 = refinement (pairs must be
 * BASE and h_new_blocks [n] must be distinct ids in [0, num_blocks) that no
 * visible logical block uses).  Each pair must be distinct, in range and
 * made of two full blocks.  Returns EKV_OK or EKV_ERR_INVALID.
 */
ekv_status ekv_check_transition(int32_t kind, const int32_t* h_pairs, int32_t n,
                                const int32_t* h_block_table, const uint8_t* h_tags,
                                const int32_t* h_seq_lens, int32_t batch, int32_t max_blocks,
                                int32_t page_size, int32_t num_blocks,
                                const int32_t* h_new_blocks);

/*
 * Device-side validation of the invariants the kernels rely on (§3.1: a
 * pair's two blocks share one fidelity, and a BASE pair is two full blocks
 * packed into one physical block; App. B.1: a transition starts from the
 * opposite state).  The kernels themselves never leave their arrays on a
 * violated invariant, but their results are then undefined; these calls
 * find such inputs without a host copy of the metadata.
 *
 * Each call re-initialises report (device int32 [2 * EKV_VIOL_COUNT], caller
 * owned) on the stream and then counts violations into it:
 *   report[k]                    number of violations of kind k
 *   report[EKV_VIOL_COUNT + k]   smallest index at which kind k occurs,
 *                                0x7fffffff if none
 * Batch indices are s * max_blocks + logical block (the checks of a whole
 * sequence -- its length, its boundaries -- use block 0); list indices are
 * the entry i of the pairs / new_blocks list.
 * Asynchronous on the stream; nothing else is written.
 *
 * With EKV_DEBUG=1 in the environment, ekv_attn_decode, ekv_attn_prefill
 * and every transition call run these checks first, synchronise the stream,
 * and return EKV_ERR_INVALID (naming the first violation) without
 * enqueuing anything else.  That mode reports into a static 48-byte device
 * array of the library (one per device; calls in this mode from several
 * host threads on one device race on it) and is meant for debugging only.
 */
enum {
  EKV_VIOL_SEQ_LEN = 0,       /* seq_lens[s] < 0, or beyond max_blocks*page_size or max_seq_len */
  EKV_VIOL_BLOCK_RANGE = 1,   /* a visible logical block maps outside [0, num_blocks) */
  EKV_VIOL_TAG_VALUE = 2,     /* a visible tag is neither TARGET nor BASE */
  EKV_VIOL_PAIR_MIXED = 3,    /* the two visible blocks of a pair have different tags */
  EKV_VIOL_BASE_PARTIAL = 4,  /* a pair executed as BASE is not two full blocks */
  EKV_VIOL_BASE_ALIAS = 5,    /* a pair executed as BASE has two different table entries */
  EKV_VIOL_MODE = 6,          /* mode / boundaries disagree with the tags (per pair), or bad boundaries (per s) */
  EKV_VIOL_LIST_RANGE = 7,    /* list pair (s, j) outside the table, or a member maps outside the pool */
  EKV_VIOL_LIST_STATE = 8,    /* list pair not TARGET (demotion) / not BASE (refinement) */
  EKV_VIOL_LIST_PARTIAL = 9,  /* list pair not two full blocks (checked when seq_lens is given) */
  EKV_VIOL_LIST_DUPLICATE = 10, /* list pair equal to an earlier entry */
  EKV_VIOL_NEW_BLOCK = 11,    /* new block out of range or equal to an earlier one; or, with
                                 seq_lens, a visible table entry holding a new block (index:
                                 the new block's list entry) */
  EKV_VIOL_COUNT = 12
};

/*
 * Checks a batch as ekv_attn_decode / ekv_attn_prefill would execute it:
 * per sequence its length; per visible logical block its table entry and
 * tag; per visible pair mixed tags, and for a pair the batch mode executes
 * as BASE (tags in GENERAL mode, boundaries in STRUCTURED mode when given,
 * none in NATIVE mode) its two full blocks and shared table entry; the
 * mode against the tags where both are given.
 * Errors: EKV_ERR_INVALID (NULL pointers, sizes), EKV_ERR_HIP.
 */
ekv_status ekv_validate_batch(const ekv_pool* pool, const ekv_batch* batch, int32_t* report,
                              hipStream_t stream);

/*
 * Checks a transition list (kind 0 demotion, 1 refinement) against the
 * device block table and tags (both [batch][max_blocks]): each pair in
 * range and mapping into the pool, in the starting state, and distinct; for
 * a refinement with new_blocks [n], each new block in range and distinct.
 * seq_lens (device [batch]) may be NULL; when given, pairs must be two full
 * blocks and no visible table entry may hold a new block.
 * Errors: EKV_ERR_INVALID (NULL pointers, sizes, kind), EKV_ERR_HIP.
 */
ekv_status ekv_validate_transition(const ekv_pool* pool, int32_t kind, int32_t n, const int32_t* pairs,
                                   const int32_t* new_blocks, const int32_t* block_table,
                                   const uint8_t* tags, const int32_t* seq_lens, int32_t batch,
                                   int32_t max_blocks, int32_t* report, hipStream_t stream);

/*
 * Pressure-aware fidelity control (§3.3, Alg. 1; defaults from App. B.1;
 * the watermark / eager-promotion / no-promotion switches of the ablations
 * in App. C.7), host only.  One scheduling step is two calls around the
 * serving scheduler; the caller applies the returned lists with
 * ekv_demote / ekv_refine (and its block allocator) and keeps the state.
 *
 * Eligible TARGET pair (s, j): both tags TARGET, both blocks full
 * (32 (j+1) <= len), sink_pairs <= j < len/32 - recent_pairs, and, when
 * h_backed (uint8 [batch][max_blocks], entry of member 0) is given, backed.
 * Demotion takes eligible pairs oldest first: ascending (j, s).  Promotion
 * takes BASE pairs (both blocks holding tokens) newest first: descending
 * j, then ascending s.  (The paper ranks by unspecified runtime signals;
 * these orders keep every sequence's BASE pairs one run next to its sink,
 * which the structured attention path serves.)
 */
#define EKV_CTRL_SHORTAGE 0          /* demote on a positive shortage (Alg. 1) */
#define EKV_CTRL_WATERMARK 1         /* demote while free blocks < watermark (ablation) */
#define EKV_CTRL_EAGER_PROMOTION 1   /* flag: promotion budget ignores the reserve (ablation) */
#define EKV_CTRL_NO_PROMOTION 2      /* flag: never promote (ablation) */

typedef struct {
  int32_t min_batch;     /* B_min: fewest pairs a triggered demotion takes (paper: 16) */
  int32_t decay;         /* lambda: reserve decay per step, in blocks (paper: 2) */
  int32_t a_max;         /* A_max: no demand probe while free blocks > a_max; < 0: always probe */
  int32_t sink_pairs;    /* pairs at the start of every sequence never demoted */
  int32_t recent_pairs;  /* last complete pairs of every sequence never demoted */
  int32_t policy;        /* EKV_CTRL_SHORTAGE or EKV_CTRL_WATERMARK */
  int32_t watermark;     /* W of EKV_CTRL_WATERMARK, in blocks */
  int32_t flags;         /* EKV_CTRL_EAGER_PROMOTION | EKV_CTRL_NO_PROMOTION */
} ekv_ctrl_config;

typedef struct {
  int32_t reserve;       /* R: decaying demotion reserve in blocks; start at 0 */
  int32_t surplus;       /* E_t of the current step (set by ekv_ctrl_demotion) */
  int32_t shortage;      /* Delta_t of the current step (set by ekv_ctrl_demotion) */
  int32_t budget;        /* P_t of the current step (set by ekv_ctrl_promotion) */
} ekv_ctrl_state;

/*
 * First half of a step, before scheduling.  demand = D_t, the blocks the
 * step needs (the paper's side-effect-free scheduler dry run, done by the
 * caller); free_blocks = F_t.  Delta_t = max(0, D_t - F_t), taken as 0
 * while F_t > a_max.  If the trigger (Delta_t, or max(0, W - F_t) under
 * EKV_CTRL_WATERMARK) is positive, writes
 * n_d = min(|eligible|, max(trigger, min_batch)) pairs (s, j) to
 * h_pairs_out [max_pairs][2] and *n_out = n_d; sets st->shortage = Delta_t
 * and st->surplus = E_t = max(0, n_d - Delta_t).  Each demoted pair frees
 * one block once the demotion completes.
 * h_tags [batch][max_blocks] and h_seq_lens [batch] are host mirrors.
 * Errors: EKV_ERR_INVALID (NULL pointers, negative sizes, a length beyond
 * max_blocks*page_size, unknown policy or flags, more than max_pairs
 * pairs chosen; the state is then unchanged).
 */
ekv_status ekv_ctrl_demotion(const ekv_ctrl_config* cfg, ekv_ctrl_state* st, int32_t demand,
                             int32_t free_blocks, const uint8_t* h_tags, const int32_t* h_seq_lens,
                             const uint8_t* h_backed, int32_t batch, int32_t max_blocks,
                             int32_t page_size, int32_t* h_pairs_out, int32_t max_pairs, int32_t* n_out);

/*
 * Second half, after the step's required scheduling and allocation, with
 * free_post = F_post free blocks.  Updates st->reserve to
 * R_t = max(0, R_{t-1} - decay) + E_t and st->budget to
 * P_t = max(0, F_post - R_t) (F_post under EKV_CTRL_EAGER_PROMOTION); then
 * writes up to min(P_t, slack) BASE pairs to h_pairs_out [max_pairs][2]
 * (none under EKV_CTRL_NO_PROMOTION).  slack = the pairs the transfer path
 * can take this step.  Each promoted pair needs one free block (the new
 * block of ekv_refine).
 * Errors: as ekv_ctrl_demotion.
 */
ekv_status ekv_ctrl_promotion(const ekv_ctrl_config* cfg, ekv_ctrl_state* st, int32_t free_post, int32_t slack,
                              const uint8_t* h_tags, const int32_t* h_seq_lens, int32_t batch,
                              int32_t max_blocks, int32_t page_size, int32_t* h_pairs_out, int32_t max_pairs,
                              int32_t* n_out);

#ifdef __cplusplus
}
#endif

#endif /* EKV_H */
