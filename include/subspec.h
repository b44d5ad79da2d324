/*
 * subspec.h -- C ABI of the MI355X (gfx950) low-bit substitute-layer library.
 *
 * SubSpec (Sec. 4.1, "Quantized Substitute Weights for Offloaded Layers") keeps a
 * GPU-resident, data-free, group-wise quantized copy of every offloaded linear
 * layer of the target model and evaluates the draft model with those copies.  The
 * draft forward (Sec. 4.2) runs on the k leaf tokens of a speculative tree, so each
 * substitute layer is a linear layer evaluated on a small token batch M against the
 * full K x N weight.  Sec. 5.1 uses 4-bit codes with groups of 64; this library
 * also takes 3- and 2-bit codes and groups of 128 (the lower bit widths are named
 * as future work in the paper's Limitations section).
 *
 * The operation, for every output row m < M and column n < N:
 *     y[m][n] = sum_k x[m][k] * s[g][n] * (q[n][k] - z[g][n]),   g = k / group
 * with bf16 activations x, unsigned `bits`-bit codes q, fp16 scale s and fp16
 * (fractional) zero-point z per group of `group` consecutive k of one column, fp32
 * accumulation and a bf16 result rounded to nearest-even.
 *
 * Conventions shared by every entry point
 *  - Pointers named "device" are HIP device memory owned by the caller; "host" are
 *    ordinary host memory.  No call frees or retains caller memory.
 *  - Calls taking a hipStream_t are asynchronous on that stream (0 = the null
 *    stream).  Argument errors are reported synchronously, before anything is
 *    enqueued.  A kernel fault surfaces at the caller's next synchronisation.
 *  - Return value: SUBSPEC_OK or a negative status; subspec_last_error() then
 *    describes the failure (thread-local, valid until the next failing call).
 *  - bits in {2,3,4}; group in {64,128}; K % 128 == 0; N % 16 == 0; M in 1..128;
 *    device pointers 16-byte aligned.
 *
 * Packed weight layout ("tile layout"; this library's own, the paper gives none)
 *  - A tile holds the codes of 16 output columns x 128 inputs.  Tile (nt, kb),
 *    nt = n / 16, kb = k / 128, starts at byte 256 * bits * (nt * (K/128) + kb), so
 *    the whole buffer is N * K * bits / 8 bytes (subspec_qpack_bytes).
 *  - A tile is 64 slices of 4*bits bytes.  Slice L (0..63) belongs to column
 *    n = 16*nt + L % 16 and holds 32 codes: for step j (0..3) and element e (0..7)
 *    the code of k = 128*kb + 32*j + 8*(L/16) + e.
 *  - The 32 codes form 16 pairs p = 4*j + e/2.  Within a slice read as
 *    little-endian 32-bit words, a pair's even-e code sits at bit offset o of a
 *    word and its odd-e code at offset o + 16 of the same word:
 *      bits 4: word p/4, o = 4*(p%4)
 *      bits 2: word p/8, o = 2*(p%8)
 *      bits 3: pairs 0..14: word p/5, o = 3*(p%5);  pair 15: bit c (c = 0,1,2) of
 *              the even code is bit 15 of word c, of the odd code bit 31 of word c.
 *    One 64-lane wavefront reading one slice per lane reads a whole tile as one
 *    contiguous run, and every pair unpacks with a shift and one and-or into two
 *    16-bit fields.
 *  - Scales and zeros are fp16 arrays [K/group][N], row-major (s[g][n] at g*N + n).
 *
 * Around the substitute linear the library also provides, each declared below with
 * its own contract: the draft-tree expansion with probability sharpening
 * (subspec_tree_*, Sec. 4.2 and App. D), the draft's tree attention over the key/value
 * cache it shares with the target (subspec_tree_attention*, Sec. 4.1), the
 * verification pass's cross-layer asynchronous weight prefetch (subspec_prefetch_*,
 * Sec. 4.3 and App. E) and the quantizer with an HQQ-style optimised zero-point
 * (subspec_quantize_hqq, Sec. 4.1 and 5.1).  The shape limits listed above are the
 * substitute linear's; the other calls state theirs.
 */
#ifndef SUBSPEC_H_
#define SUBSPEC_H_

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

enum subspec_status {
  SUBSPEC_OK = 0,
  SUBSPEC_EINVAL = -1,       /* bad argument (null/misaligned pointer, bad size) */
  SUBSPEC_EUNSUPPORTED = -2, /* well-formed but outside bits/group/M/N/K support */
  SUBSPEC_EHIP = -3,         /* a HIP runtime call or kernel launch failed        */
  SUBSPEC_ECAPTURE = -4      /* the call needs to grow its workspace while the
                                stream is being captured; call subspec_reserve()
                                before capturing                                  */
};

/* Kernel paths (subspec_plan.path, subspec_qlinear_path's `path`). */
enum subspec_path {
  SUBSPEC_PATH_AUTO = 0, /* let subspec_qlinear_plan choose                        */
  SUBSPEC_PATH_GEMV = 1, /* VALU dot products; the four 16-lane quarters of a
                            wavefront split K and are summed with lane shuffles,
                            per-group sums of x reduced with DPP; M <= 8          */
  SUBSPEC_PATH_MFMA = 2, /* bf16 matrix cores on unpacked code tiles; any M; the
                            plan picks the instruction shape (below)             */
  SUBSPEC_PATH_MFMA16 = 3, /* MFMA path on 16x16x32 instructions (row tiles of 16) */
  SUBSPEC_PATH_MFMA32 = 4  /* MFMA path on 32x32x16 instructions, 128 rows (four
                              row blocks of 32), or 64 where M <= 64 and the
                              eight-wavefront kernel runs; rows past M are padding */
};

/* Launch configuration chosen for one qlinear call (host-side description). */
typedef struct subspec_plan {
  int path;            /* SUBSPEC_PATH_GEMV or SUBSPEC_PATH_MFMA                  */
  int mfma_rows;       /* MFMA path: 16 (16x16x32 bf16 instructions) or 32
                          (32x32x16 bf16); 0 on the GEMV path.  The automatic
                          choice takes 32 for M > 64 on launches that either fill
                          every CU with whole 128-column groups or split a K of at
                          least 16384, and for 32 < M <= 64 on launches whose
                          256-column groups cover three quarters of the CUs with K
                          unsplit or whose K is at least 16384 (measured on the
                          Qwen2.5 shapes)                                        */
  int rows;            /* rows computed per workgroup (M rounded up; with row_blocks
                          = 2, half of that)                                     */
  int tiles_per_wave;  /* 16-column tiles each wavefront owns                     */
  int waves;           /* wavefronts per workgroup                                */
  int chunk_blocks;    /* 128-k blocks staged in LDS per step                     */
  int ring_chunks;     /* MFMA path: chunks of weights in each wavefront's register
                          ring (0 = the kernel's default; GEMV: ring stages)     */
  int col_groups;      /* column groups (waves / teams * tiles_per_wave * 16 columns each) */
  int full_groups;     /* column groups [0, full_groups) run whole, one workgroup
                          each; the others are split along K                    */
  int splits;          /* workgroups per split column group; 1 = no partial sums  */
  int blocks_per_split;/* 128-k blocks per split                                  */
  int grid;            /* workgroups of one row block =
                          full_groups + (col_groups - full_groups) * splits      */
  size_t workspace_bytes; /* device scratch the call uses: 64 KiB of completion
                             counters, the 32x32 kernel's per-group sums of x, and
                             the fp32 partial sums of split column groups (0 when
                             none of these is needed) */
  int teams;           /* 32-row MFMA tiles: wavefront teams per workgroup that split
                          its k-blocks between them (1, or 2: two teams of four on
                          the same columns, summed in LDS; the automatic choice on
                          a K of at least 16384 from M = 33); a workgroup covers
                          waves / teams * tiles_per_wave * 16 columns             */
  int row_blocks;      /* 16-row MFMA tiles: the rows in row_blocks blocks of `rows`
                          rows each (1 or 2), each block of workgroups an independent
                          launch along grid y with its own partial sums and
                          completion counters.  The automatic choice takes 2 for
                          M > 32 on launches whose column groups number fewer than
                          the CUs and whose K is under 16384 (q|k|v and o shapes) */
} subspec_plan;

/* Bytes of the packed code buffer for an N x K projection.  0 on bad arguments. */
size_t subspec_qpack_bytes(int bits, int N, int K);

/* Quantize fp32 weights per group with the min/max asymmetric rule (the paper's
 * data-free substitute construction, Sec. 4.1; the rule itself is this library's
 * reading, the paper names HQQ without its algorithm):
 *   s = (wmax - wmin) / (2^bits - 1) in float64;  s16 = fp16(s) nearest-even;
 *   z16 = fp16(-wmin / s16);  q = clamp(rint(w / s16 + z16), 0, 2^bits - 1),
 * every step in float64 (ties to even); a group with wmax == wmin or s16 == 0 gets
 * s16 = 1, z16 = fp16(-wmin), q = 0.
 *   w      device fp32 [N][K] row-major (read only)
 *   codes  device uint8 [N][K] row-major, one code per byte (written)
 *   scales, zeros  device fp16 [K/group][N] (written)
 * Needs K % group == 0 and N >= 1; K need not be a multiple of 128 here. */
int subspec_quantize(const float* w, int bits, int group, int N, int K,
                     uint8_t* codes, uint16_t* scales, uint16_t* zeros,
                     hipStream_t stream);

/* Same contract and outputs as subspec_quantize, with the zero of every group
 * optimised as in HQQ, the data-free quantizer SubSpec uses for its substitutes
 * (Sec. 4.1; 4-bit, groups of 64, Sec. 5.1).  The paper gives no algorithm; this
 * follows the cited half-quadratic quantization work: the scale stays the min/max
 * scale; from the min/max zero, rounds of (quantize with z; e = sign(x) max(|x| -
 * |x|^(p-1)/beta, 0) for x = w - s (q - z); z = mean(q - (w - e) / s)) with p = 0.7,
 * beta = 10 growing by 1.01 per round, at most 20 rounds, keep the zero with the
 * smallest sum |w - s (q - z)| and stop at the first round that does not improve it.
 * The best zero (fp16) replaces the min/max zero only if it is still better in fp16,
 * so no group's error grows.  float64 throughout, sums in index order. */
int subspec_quantize_hqq(const float* w, int bits, int group, int N, int K,
                         uint8_t* codes, uint16_t* scales, uint16_t* zeros,
                         hipStream_t stream);

/* Pack one-byte codes (device uint8 [N][K], each < 2^bits) into the tile layout
 * above (device, subspec_qpack_bytes() bytes, written).  Codes with bits above
 * `bits` set are masked off. */
int subspec_qpack(const uint8_t* codes, int bits, int N, int K, void* qweight,
                  hipStream_t stream);

/* Same as subspec_qpack on host memory, synchronous, no GPU needed. */
int subspec_qpack_host(const uint8_t* codes, int bits, int N, int K, void* qweight);

/* The substitute layer (Sec. 4.1): y = x * dequant(qweight, scales, zeros)^T.
 *   x        device bf16 [M][K] row-major
 *   qweight  device, tile layout, subspec_qpack_bytes(bits, N, K) bytes
 *   scales   device fp16 [K/group][N]
 *   zeros    device fp16 [K/group][N]
 *   y        device bf16 [M][N] row-major, fully overwritten
 * x and y must not overlap each other or the weights.  Uses the library's
 * per-device workspace (see subspec_reserve: the call may grow it); calls that
 * overlap in time on one device (different streams) must not share it, so
 * serialise them. */
int subspec_qlinear(const void* x, const void* qweight, const void* scales,
                    const void* zeros, int bits, int group, int M, int N, int K,
                    void* y, hipStream_t stream);

/* For callers that cannot allocate device memory (code under HIP graph capture,
 * serving loops, harnesses that forbid hipMalloc): subspec_qlinear's contract, with
 * the call's scratch (split-K completion counters, per-group sums of x, partial sums)
 * taken from a fixed array of SUBSPEC_NOALLOC_SCRATCH_BYTES per device inside the
 * library instead of the growable workspace.  The call never allocates or frees
 * memory.  The plan is subspec_qlinear's, except that the split count is reduced where
 * the partial sums would not fit: when subspec_qlinear_plan's workspace_bytes is at
 * most SUBSPEC_NOALLOC_SCRATCH_BYTES the results are bit-identical to subspec_qlinear's,
 * otherwise they differ in the order of fp32 additions only.  Shapes that need more
 * scratch even unsplit return SUBSPEC_EUNSUPPORTED.  The first call on a device looks
 * the array up and zeroes its counters on `stream` (waiting for that stream); that
 * first call must not be captured (SUBSPEC_ECAPTURE), later calls may be.  All calls
 * on one device share its array, which keeps the last call's contents: calls that
 * overlap in time on one device (different streams, concurrent graph replays) race
 * and must be serialised.  The array stays allocated until the process ends. */
#define SUBSPEC_NOALLOC_SCRATCH_BYTES ((size_t)32 << 20)
int subspec_qlinear_noalloc(const void* x, const void* qweight, const void* scales,
                            const void* zeros, int bits, int group, int M, int N, int K,
                            void* y, hipStream_t stream);

/* subspec_qlinear with an explicit kernel path (SUBSPEC_PATH_*): for tests and
 * A/B measurements.  SUBSPEC_PATH_GEMV requires M <= 8.  All paths compute the same
 * function; they differ in the order of the fp32 additions only. */
int subspec_qlinear_path(const void* x, const void* qweight, const void* scales,
                         const void* zeros, int bits, int group, int M, int N, int K,
                         void* y, int path, hipStream_t stream);

/* Host only, no GPU needed: validate the shape and fill *plan with the launch
 * configuration subspec_qlinear_path would use for `path` (AUTO allowed). */
int subspec_qlinear_plan(int M, int N, int K, int bits, int group, int path,
                         subspec_plan* plan);

/* Materialise the dequantized weights from the packed layout (the same unpacking
 * code the qlinear kernels use):
 *   w_f32[n][k]  = fma(q, s, -s*z) in fp32, which equals s*(q - z) rounded once
 *                  (s*z of two fp16 values is exact in fp32);
 *   w_bf16[n][k] = that fp32 value rounded to bf16, nearest-even.
 * Either output pointer may be null.  Outputs are device [N][K] row-major. */
int subspec_qdequant(const void* qweight, const void* scales, const void* zeros,
                     int bits, int group, int N, int K, float* w_f32,
                     uint16_t* w_bf16, hipStream_t stream);

/* One projection of a decoder layer for the per-layer launch plan: the draft model
 * evaluates, per layer, q|k|v (one launch over concatenated columns: they share x),
 * o, gate|up (concatenated, they share x) and down -- 7 substitute projections in 4
 * launches.  Concatenating along N is done by the caller before packing (codes
 * [N1+N2][K], scales and zeros [K/group][N1+N2]); quantization is per column, so the
 * fused projection is exactly the separate ones side by side. */
typedef struct subspec_proj {
  const void* x;        /* device bf16 [M][K]                         */
  const void* qweight;  /* device, tile layout                        */
  const void* scales;   /* device fp16 [K/group][N]                   */
  const void* zeros;    /* device fp16 [K/group][N]                   */
  void* y;              /* device bf16 [M][N]                         */
  int N, K;
} subspec_proj;

/* Run nproj substitute projections in order on `stream` (each one subspec_qlinear;
 * the automatic plan per shape).  All share bits, group and M. */
int subspec_stack_forward(const subspec_proj* projs, int nproj, int bits, int group, int M,
                          hipStream_t stream);

/* A captured launch sequence (HIP graph) of subspec_stack_forward. */
typedef struct subspec_graph subspec_graph;

/* Capture subspec_stack_forward(projs, ...) on `stream` (which must not be the null
 * stream) into a graph and instantiate it.  The workspace the sequence needs is
 * reserved before capture; the graph keeps using that buffer, which stays allocated
 * until the graph is destroyed even if later calls grow the workspace.  The graph keeps the pointers of `projs` (not the array):
 * replays read and write the same buffers. */
int subspec_stack_capture(const subspec_proj* projs, int nproj, int bits, int group, int M,
                          hipStream_t stream, subspec_graph** graph);

/* Replay a captured sequence on `stream` (asynchronous). */
int subspec_graph_launch(subspec_graph* graph, hipStream_t stream);

/* Release a captured sequence (synchronises the device).  Destroying the device's
 * last live graph frees the workspace buffers retired while graphs were alive. */
int subspec_graph_destroy(subspec_graph* graph);

/* Draft-tree expansion with probability sharpening (Sec. 4.2 "Constructing Deep
 * Context-Aware Dynamic Draft Tree" and "Draft Probability Sharpening", App. D): after
 * a draft pass, leaf i of the tree has logits l_i over the vocabulary and a path
 * score s_i.  Every candidate (leaf i, token v) scores
 *     score(i, v) = s_i + log softmax(l_i / T)(v)
 * -- the logarithm of the product of the parent's path score and the sharpened
 * conditional probability (the paper uses T = 0.2 for greedy decoding; path scores
 * are carried as natural logarithms, 0 at the root) -- and the k best candidates
 * over all leaves are the next leaves.  Order: larger score first, ties broken by
 * the smaller flat index i * V + v.  fp32 arithmetic; every reduction in a fixed
 * order, so repeated calls give identical results.
 *   logits       device bf16 [R][V] row-major, finite values, 16-byte aligned
 *   parent_logp  device fp32 [R]: s_i
 *   parent_out   device int32 [k]: leaf index i of each winner, best first
 *   token_out    device int32 [k]: token v
 *   score_out    device fp32 [k]: score(i, v)
 * Needs 1 <= R <= 1024, V a positive multiple of 8, R * V < 2^31, 1 <= k <= 32,
 * k <= R * V, T > 0 and 1/T finite.  Uses the library's per-device workspace
 * (subspec_tree_workspace_bytes bytes; see subspec_reserve); like subspec_qlinear,
 * calls that overlap in time on one device must be serialised. */
int subspec_tree_expand(const void* logits, const float* parent_logp, int R, int V,
                        float temperature, int k, int* parent_out, int* token_out,
                        float* score_out, hipStream_t stream);

/* Workspace bytes subspec_tree_expand needs for (R, V, k); 0 on bad arguments. */
size_t subspec_tree_workspace_bytes(int R, int V, int k);

/* Launch shape subspec_tree_expand uses for (R, V, k), computed on the host with no
 * device access: every row is cut into `chunks` slices of `chunk_len` logits (the
 * last may be shorter), one 256-thread workgroup each, so the grid has R * chunks
 * workgroups; `list_len` is the per-thread candidate list length (8, 16 or 32, the
 * kernel's template argument).  Outputs are host pointers.  Returns SUBSPEC_OK,
 * SUBSPEC_EINVAL for a null output, or SUBSPEC_EUNSUPPORTED for an (R, V, k) that
 * subspec_tree_expand would reject. */
int subspec_tree_plan(int R, int V, int k, int* chunks, int* chunk_len, int* list_len);

/* Tree attention of one decoder layer in one draft pass, over the key/value cache the
 * draft model shares with the target (SubSpec Sec. 4.1, "Shared KV-Cache"; the tree
 * masks of tree decoding, Sec. 2 and Sec. 4.2).  M new tree tokens with Hq query
 * heads (head dimension 128) grouped onto Hkv key/value heads (query head h reads
 * key/value head h / (Hq / Hkv)) attend, with scores q.k * scale and a softmax, to
 *   - every committed cache position 0 .. P - 1,
 *   - cache position P + j (j < T: tree tokens of earlier passes; j = T + i: new
 *     token i) when bit j of their mask row is set.
 * The new keys and values are appended to the cache at P + T .. P + T + M - 1 (the
 * target's verification later overwrites them); within this call the new tokens'
 * keys and values are read from k_new / v_new.  A query with no visible position
 * gets zeros.
 *   q        device bf16 [M][Hq][128] (positions already rotated)
 *   k_cache  device bf16 [Hkv][S][128], one layer; rows P + T .. P + T + M - 1 are
 *   v_cache  overwritten with k_new / v_new, all others are only read
 *   k_new    device bf16 [M][Hkv][128]
 *   v_new    device bf16 [M][Hkv][128]
 *   mask     device uint32 [M][W], W = ceil((T + M) / 32); bit j % 32 of word j / 32
 *            of row i allows tree position j to token i
 *   out      device bf16 [M][Hq][128]
 * Needs Hkv >= 1, Hq a multiple of Hkv, 1 <= M and (Hq / Hkv) * M <= 64, P, T >= 0,
 * P + T + M <= S, M * W <= 2048, a finite scale; q, caches, new rows and out 16-byte
 * aligned, mask 4-byte aligned; out must not overlap the inputs.  Two kernels on
 * `stream` (partial outputs per key range, then their combination and the append);
 * workspace as for subspec_qlinear (subspec_tree_attention_workspace_bytes). */
int subspec_tree_attention(const void* q, void* k_cache, void* v_cache, const void* k_new,
                           const void* v_new, const uint32_t* mask, int M, int Hq, int Hkv,
                           int S, int P, int T, float scale, void* out, hipStream_t stream);

/* Workspace bytes subspec_tree_attention needs; 0 on bad arguments. */
size_t subspec_tree_attention_workspace_bytes(int M, int Hq, int Hkv, int P, int T);

/* Launch shape of subspec_tree_attention, on the host: the P + T + M keys of each
 * key/value head are cut into `splits` ranges of `tiles_per_split` tiles of 32 keys;
 * the first kernel runs splits x Hkv workgroups.  Returns SUBSPEC_OK, SUBSPEC_EINVAL
 * for a null output or SUBSPEC_EUNSUPPORTED for shapes subspec_tree_attention would
 * reject (S is not checked here). */
int subspec_tree_attention_plan(int M, int Hq, int Hkv, int P, int T, int* splits,
                                int* tiles_per_split);

/* Cross-layer asynchronous weight prefetch for the verification pass (SubSpec
 * Sec. 4.3 "Asynchronous Data Transfer", App. E): while the GPU computes with one
 * offloaded tensor, the next ones are copied from pinned host memory into a fixed
 * ring of reused device buffers (peak memory does not grow with the model), across
 * decoder-layer boundaries.
 *
 * A prefetcher owns `slots` device buffers of `slot_bytes` each on the device current
 * at creation, and one copy stream (default priority).  Tickets 0, 1, 2, ... are
 * handed out in order; ticket t uses slot t % slots.  Per ticket:
 *   begin    enqueue the host-to-device copy on the copy stream, after the work that
 *            released the slot's previous ticket (an event on the releasing stream);
 *   acquire  make `compute` wait for that copy; returns the slot's device pointer,
 *            valid for work enqueued on `compute` until the ticket is released;
 *   release  record, on `compute`, that all work using the slot is enqueued.
 * begin fails with SUBSPEC_EINVAL while the slot's previous ticket is not released
 * (there is no host-side wait), so a missing release is an error, never a race.
 * Host sources must be pinned (hipHostMalloc, or torch's pin_memory); the copies are
 * asynchronous and the host buffer must stay unchanged until the compute stream has
 * passed the acquire.  Calls on one prefetcher must not overlap in time. */
typedef struct subspec_prefetch subspec_prefetch;
int subspec_prefetch_create(size_t slot_bytes, int slots, subspec_prefetch** out);
int subspec_prefetch_destroy(subspec_prefetch* pf); /* waits for its copies */
int subspec_prefetch_begin(subspec_prefetch* pf, const void* host_src, size_t bytes,
                           long long* ticket);
int subspec_prefetch_acquire(subspec_prefetch* pf, long long ticket, hipStream_t compute,
                             void** dev_ptr);
int subspec_prefetch_release(subspec_prefetch* pf, long long ticket, hipStream_t compute);

/* The per-device workspace.  subspec_qlinear, subspec_tree_expand and
 * subspec_tree_attention share one device buffer per device: its first 64 KiB are
 * split-K completion counters (zero between calls), the rest is scratch for the call
 * in flight.  A call that needs more than the buffer holds grows it: hipMalloc of a
 * buffer at least twice as large, its counters zeroed on the call's stream, and a
 * wait on that stream only (never on the whole device).  The old buffer is retired,
 * not freed, because kernels queued on other streams or captured graphs
 * (subspec_stack_capture) may still use it.  Retired buffers are freed by
 * subspec_reserve while no captured graph is alive on the device, and when the
 * device's last captured graph is destroyed; both synchronise the device first.  A
 * call made after subspec_reserve(bytes) with a need of at most `bytes` neither
 * allocates, frees nor synchronises.
 *
 * subspec_reserve: grow the calling device's workspace to at least `bytes` now
 * (synchronous; may call hipMalloc) and free retired buffers as above, so that later
 * calls, e.g. under stream capture, need not allocate. */
int subspec_reserve(size_t bytes);

/* Current state of the calling device's workspace: its size in bytes, the number of
 * retired buffers still held, and how many buffers it has allocated so far.  Any
 * output pointer may be null.  Host only; no GPU work. */
int subspec_workspace_info(size_t* bytes, int* retired, unsigned long long* allocations);

/* Description of the last failure on this thread ("" if none). */
const char* subspec_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* SUBSPEC_H_ */
