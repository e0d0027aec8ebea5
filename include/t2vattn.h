/*
 * libt2vattn: bidirectional multi-head self-attention, forward and backward,
 * over packed variable-length token sequences, for AMD MI355X (gfx950).
 *
 * The operation (paper Section III, Observation 2): every clip is one sequence
 * of 3D latent patches, and each token attends to every token of its own clip
 * (full, non-causal self-attention), at O(L^2) cost per clip -- the alpha_2 *
 * B * S^2 term of the DiT latency model, Eq. (9). Clips are packed back to back
 * along the token axis and described by cu_seqlens, so clips of different
 * resolution and duration share one call without padding (Section II-B
 * contrasts padding, packing and bucketing). The training step runs this
 * operation forward and backward (Fig. 1 caption: DiT backward pass).
 *
 * For clip s (tokens cu[s] .. cu[s+1]-1, length L = cu[s+1]-cu[s]) and head h,
 * with Q, K, V, dO the [L, D] slices:
 *   S = scale * Q K^T;  P = softmax over each row of S;  out = P V;
 *   lse_i = ln(sum_j exp(S_ij))   (natural log, the row normaliser);
 *   Delta_i = sum_d dO_id out_id;  dP = dO V^T;  dS = P * (dP - Delta);
 *   dq = scale * dS K;  dk = scale * dS^T Q;  dv = P^T dO.
 * Gradients are those of the scalar <dout, out>; lse is not differentiated.
 *
 * Layout. Every tensor is row-major and contiguous, "THD": element (t, h, d)
 * of a [T, H, D] tensor sits at ((t * H) + h) * D + d. q, k, v, out, dout, dq,
 * dk, dv are bfloat16 (passed as void*). lse is float32 laid out [H, T]:
 * element (h, t) at h * T + t; delta_ws holds two such arrays. T = cu_seqlens[nseq].
 *
 * Ownership. The caller owns every buffer. Tensor pointers are device
 * pointers; cu_seqlens is a HOST pointer (the tile scheduler runs on the
 * host). The library keeps only a cache of device work lists keyed by the
 * contents of cu_seqlens (released by t2v_release_cache). It holds up to 64;
 * the call that adds one more releases the least recently used. List memory
 * comes from pooled device and pinned chunks; a released list's memory is
 * reused only after the launches that read it have finished (events recorded
 * on their streams), so no call waits for the device.
 *
 * Tiles. The forward and dQ kernels own 256-query tiles (8 waves, one workgroup per CU)
 * or 128-query tiles (4 waves, two or three per CU): narrow tiles at head_dim 64, and at
 * 128 when the work-weighted key length sum(Lq Lk^2) / sum(Lq Lk) is at most 1,536 (forward)
 * or 8,192 (dQ), where they were measured faster, or when the host's list-scheduling model
 * predicts that the wide tiles would leave CUs idle in a part-empty last round (packs with
 * few tiles per CU, e.g. a long clip at a few heads). The choice is made once per new work
 * list. Both shapes give bitwise-equal results. The dK/dV kernel owns 128-key tiles and loops over the
 * sequence's queries; when the costliest such loop exceeds an even share of the work over
 * the GPU's CUs (few, short key segments against long query segments, as in
 * cross-attention to text), the loops are cut into pieces of at least 2048 queries whose
 * fp32 partial sums are kept in dq's memory and added in piece order before the dQ kernel
 * overwrites dq. Results stay deterministic; they differ from the unsplit order only by
 * rounding.
 *
 * Environment. T2V_ORDER=natural schedules tiles in pack order instead of longest clip
 * first (for ablations); T2V_QTILE=wide or narrow forces the forward / dQ tile shape and
 * T2V_SPLIT=off disables the dK/dV loop split (ablations and tests); T2V_PERSISTENT=1 runs the
 * forward and dK/dV kernels on a persistent grid (as many workgroups as the GPU holds at once,
 * each striding over the work list; bitwise-equal results, measured ~1% slower, so off by
 * default). T2V_LOG=1 prints one
 * line to stderr per new work list: its items, the host's predicted list-scheduling
 * makespan and its lower bound, and the loop split if any. T2V_TEST_FAIL_ALLOC=1 makes
 * building a new work list fail with T2V_ERR_OOM, for testing that path.
 *
 * Threads. Calls from several host threads, on one stream or several, are
 * safe: the cache is guarded by a mutex and a work list stays allocated while
 * any call that looked it up is still enqueueing its launches.
 *
 * Errors. Every function returns a t2v_status. Arguments are validated before
 * anything is launched, so a rejected call writes nothing. Execution is
 * asynchronous on `stream` (a hipStream_t; NULL is the default stream). A
 * kernel launch failure returns T2V_ERR_HIP. t2v_last_error() describes the
 * last non-OK status of the calling thread. No C++ exception crosses the ABI.
 * T = 0 returns T2V_OK without launching anything; zero-length clips are
 * skipped. Calls on different streams may run concurrently.
 *
 * Checked library. libt2vattn_checked.so exports the same calls, built from the same
 * sources with bounds checks, for debugging: before any kernel runs, every work list is
 * checked on the host against cu_seqlens (each tile inside its clip, each looped-over row
 * inside the same clip, heads and partial slots in range); on the device every row a kernel
 * copies into LDS is checked against its clip (a failing row is not copied); and each call
 * waits for its kernels before returning. A violation returns T2V_ERR_BOUNDS and
 * t2v_last_error() names the work item, or the kernel, workgroup and row. Calls into it are
 * serialised. T2V_CHECK_CANARY=n takes n rows off every bound the kernels check, so correct
 * kernels report their clips' last rows: a way to see that the checks report. Its results
 * equal the unchecked library's bitwise.
 */
#ifndef T2VATTN_H
#define T2VATTN_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  T2V_OK = 0,
  T2V_ERR_INVALID_ARG = 1, /* bad pointer, size, cu_seqlens, scale or aliasing */
  T2V_ERR_UNSUPPORTED = 2, /* head_dim other than 64 or 128 */
  T2V_ERR_HIP = 3,         /* a HIP runtime call or kernel launch failed */
  T2V_ERR_OOM = 4,         /* the work-list cache could not allocate */
  T2V_ERR_BOUNDS = 5       /* checked library only: a work item, or a row a kernel copies,
                              lies outside its clip (see "Checked library" below) */
} t2v_status;

/* Tile orders for the scheduler (see t2v_build_worklist). */
typedef enum {
  T2V_ORDER_NATURAL = 0,      /* clip, head, tile in pack order */
  T2V_ORDER_LONGEST_FIRST = 1 /* clips by length descending; (clip, head) tiles kept adjacent;
                                 dealt to the 8 XCDs in cost-balanced contiguous runs */
} t2v_order;

/* Forward pass: out = softmax(scale * q k^T) v per clip and head, and lse.
 *   q, k, v    device bf16 [T, H, D], 16-byte aligned, read only
 *   cu_seqlens host int32 [nseq + 1]: cu[0] = 0, non-decreasing, cu[nseq] = T < 2^31
 *   nseq       number of clips (>= 0); heads = H (>= 1); head_dim = D in {64, 128};
 *              H * D <= 2^22 and T * H * D <= 2^40, else T2V_ERR_INVALID_ARG
 *   scale      finite multiplier of q k^T (1/sqrt(D) in the usual case)
 *   out        device bf16 [T, H, D], written; must not overlap any input
 *   lse        device fp32 [H, T], written; natural-log row normaliser
 *   stream     hipStream_t to launch on
 */
int t2v_attn_fwd(const void* q, const void* k, const void* v,
                 const int32_t* cu_seqlens, int nseq, int heads, int head_dim, float scale,
                 void* out, float* lse, void* stream);

/* Backward pass for the loss <dout, out>: dq, dk, dv.
 *   q, k, v, cu_seqlens, nseq, heads, head_dim, scale   as passed to t2v_attn_fwd
 *   out, lse   the forward outputs for the same inputs (device, read only)
 *   dout       device bf16 [T, H, D], the gradient of the loss w.r.t. out
 *   dq, dk, dv device bf16 [T, H, D], written; must not overlap each other or any input
 *              (dq's memory also serves as scratch during the call, see Tiles above)
 *   delta_ws   device fp32 [2, H, T], caller-owned scratch (8 * H * T bytes): receives
 *              -Delta = -rowsum(dout * out) in [0] and lse * log2(e) in [1]
 *   stream     hipStream_t to launch on
 * Deterministic: no atomics; repeated calls give bitwise-equal results.
 */
int t2v_attn_bwd(const void* q, const void* k, const void* v,
                 const void* out, const float* lse,
                 const int32_t* cu_seqlens, int nseq, int heads, int head_dim, float scale,
                 const void* dout, void* dq, void* dk, void* dv, float* delta_ws,
                 void* stream);

/* Backward pass that allocates nothing, for callers that cannot allocate device memory
 * (code under stream capture, tight serving loops, harnesses that forbid allocation).
 * Arguments, results and errors are those of t2v_attn_bwd without delta_ws: the Delta / lse
 * scratch (8 * heads * T bytes) and the dK/dV and dQ work lists (32 bytes per work item,
 * built on the host at every call, not cached) are kept in one static 64 MiB device array
 * of the library, one per GPU, held until the process ends. No hipMalloc, hipHostMalloc or
 * other device allocation is made; the work lists are copied from host memory with
 * hipMemcpyAsync on `stream`, which for a pageable source makes the call wait for that copy.
 *   Limit: a call needing more than 64 MiB (8 * heads * T plus the lists: about
 *   heads * T <= 8e6 tokens x heads) returns T2V_ERR_INVALID_ARG before any launch.
 *   Every call on a GPU shares the array: calls on one stream are ordered by it, but calls
 *   that overlap on one GPU (other streams, other threads) race and must not be made.
 * Results are bitwise equal to t2v_attn_bwd's for the same inputs. */
int t2v_attn_bwd_noalloc(const void* q, const void* k, const void* v,
                         const void* out, const float* lse,
                         const int32_t* cu_seqlens, int nseq, int heads, int head_dim, float scale,
                         const void* dout, void* dq, void* dk, void* dv, void* stream);

/* Cross-attention: queries and keys from separate token streams, e.g. a clip's video tokens
 * attending to its text tokens. The paper's Wan2.1 model uses self- and cross-attention
 * (Section V-A), the DiT is conditioned on text (Section II-A), and text sequences are short,
 * typically under 256 tokens (Section IV-B footnote). For sequence s, queries are rows
 * cu_seqlens_q[s] .. cu_seqlens_q[s+1] - 1 of q (and of out, lse, dout, dq), keys and values
 * are rows cu_seqlens_k[s] .. cu_seqlens_k[s+1] - 1 of k and v (and of dk, dv); each query
 * attends to every key of its sequence. Everything else is as in t2v_attn_fwd / t2v_attn_bwd,
 * with Tq = cu_seqlens_q[nseq] and Tk = cu_seqlens_k[nseq]:
 *   q, out, dout, dq   device bf16 [Tq, H, D];   k, v, dk, dv   device bf16 [Tk, H, D]
 *   lse                device fp32 [H, Tq];      delta_ws       device fp32 [2, H, Tq]
 *   cu_seqlens_q, cu_seqlens_k   HOST int32 [nseq + 1] each, both validated as cu_seqlens
 * A sequence must have both queries and keys, or neither (a query without keys has no
 * softmax): otherwise T2V_ERR_INVALID_ARG. Passing the same array twice is self-attention,
 * identical to t2v_attn_fwd / t2v_attn_bwd. Deterministic, like them. */
int t2v_attn_fwd_qk(const void* q, const void* k, const void* v,
                    const int32_t* cu_seqlens_q, const int32_t* cu_seqlens_k, int nseq,
                    int heads, int head_dim, float scale, void* out, float* lse, void* stream);

int t2v_attn_bwd_qk(const void* q, const void* k, const void* v,
                    const void* out, const float* lse,
                    const int32_t* cu_seqlens_q, const int32_t* cu_seqlens_k, int nseq,
                    int heads, int head_dim, float scale,
                    const void* dout, void* dq, void* dk, void* dv, float* delta_ws,
                    void* stream);

/* Thread-local message describing the last non-OK status of this thread. */
const char* t2v_last_error(void);

/* Waits for the device, then frees every cached work list. Safe to call at any time. */
void t2v_release_cache(void);

/* Host-only scheduler, exposed for testing. Builds the work list the kernels use for
 * tiles of `block` rows: each item is 4 int32 {row0 of the clip, clip length L,
 * first row of the tile within the clip, head}. Clips of length 0 give no items.
 *   order       a t2v_order
 *   items_out   host int32 [capacity * 4], or NULL to query the count only
 *   n_items_out receives the number of items
 * Returns T2V_ERR_INVALID_ARG if capacity is too small (n_items_out is still set).
 */
int t2v_build_worklist(const int32_t* cu_seqlens, int nseq, int heads, int block, int order,
                       int32_t* items_out, int capacity, int* n_items_out);

/* Host-only: the predicted makespan of a work list on `slots` identical workers, in units
 * of (rows x keys) tile cost, when items are taken in list order by the next free worker
 * (greedy list scheduling), plus the lower bound max(total / slots, largest item).
 * `items` holds n_items items of 4 int32 as returned by t2v_build_worklist. */
int t2v_plan_makespan(const int32_t* items, int n_items, int block, int slots,
                      double* makespan_out, double* lower_bound_out);

/* Cascade scheduling (paper Section IV-A, Eqs. (1)-(7)), host-only. Cascades c = 0..n-1
 * form a DAG given by predecessor lists in CSR form: the direct predecessors of c are
 * pred_idx[pred_ptr[c] .. pred_ptr[c+1]-1] (pred_ptr[0] = 0, non-decreasing; indices in
 * 0..n-1, no self-loops; a cycle is T2V_ERR_INVALID_ARG). A schedule gives each cascade a
 * parallel degree k_c (GPUs) and a launch time s_c >= the end of every predecessor; the
 * degrees of the cascades running at any time sum to at most n_gpus.
 *
 * t2v_list_schedule: for fixed degrees (degree[c] in 1..n_gpus) and latencies (latency[c],
 * finite, >= 0), the critical-path list schedule: the ready cascade with the longest chain
 * of latencies from it to the end of the graph goes first, at the earliest time its
 * predecessors have ended and its GPUs are free for its whole latency. Writes start_out[n]
 * (host doubles) and the makespan. */
int t2v_list_schedule(int n_cascades, const int32_t* pred_ptr, const int32_t* pred_idx,
                      const int32_t* degree, const double* latency, int n_gpus,
                      double* start_out, double* makespan_out);

/* t2v_plan_cascades: chooses the degrees too (Alg. 1: a genetic algorithm whose fitness is
 * t2v_list_schedule's makespan). degrees[n_degrees] is the set K (each >= 1); latency and
 * mem are host doubles [n_cascades][n_degrees]: L_{c,k} and Mem_{c,k}. A degree is feasible
 * for c when Mem_{c,k} <= mem_cap (W) and k <= n_gpus; a cascade with none is
 * T2V_ERR_INVALID_ARG. GA hyper-parameters: population >= 2, generations >= 0, mutation
 * rate in [0, 1], 0 <= elite <= population; seed makes the result reproducible. Writes the
 * best schedule found: degree_out[n] (the chosen k), start_out[n], makespan_out. */
int t2v_plan_cascades(int n_cascades, const int32_t* pred_ptr, const int32_t* pred_idx,
                      int n_degrees, const int32_t* degrees, const double* latency,
                      const double* mem, double mem_cap, int n_gpus,
                      int population, int generations, double mutation, int elite, uint64_t seed,
                      int32_t* degree_out, double* start_out, double* makespan_out);

/* Per-kernel timing, for measurement. While enabled, every kernel launch is bracketed by
 * two HIP events recorded on the launch stream. t2v_kernel_times waits for the recorded
 * events, returns the summed elapsed milliseconds and the launch count of each kernel since
 * the previous read (slots: 0 forward, 1 backward Delta, 2 backward dK/dV, 3 backward dQ),
 * and forgets them. Enabling or disabling also forgets. Calls overlapping with launches on
 * other host threads are serialised by a mutex.
 *   ms_out     host double[4];  counts_out host int[4] */
int t2v_timing_enable(int on);
int t2v_kernel_times(double* ms_out, int* counts_out);

/* Per-workgroup trace, for measurement: the single-GPU analogue of the per-rank balance
 * metric of the case study (Section V-E), i.e. per-CU busy time and its coefficient of
 * variation. While armed, every forward, dK/dV and dQ kernel launch takes the next n_items
 * records of dev_records, one per workgroup in work-list order, each four uint64:
 * {CU id, start, end, kernel slot}; CU id = (XCC_ID << 16) | bits 8..15 of HW_ID, start
 * and end on the constant 100 MHz device clock, slot 0 forward, 2 dK/dV, 3 dQ. A launch
 * whose records do not fit runs untraced and is counted as overflowed. Tracing does not
 * change any result.
 *   dev_records  device unsigned long long[4 * capacity], 8-byte aligned, caller-owned;
 *                NULL (with capacity 0) disarms
 *   t2v_trace_set resets the count; t2v_trace_count returns the records taken so far and
 *   the number of launches that did not fit.
 * Invalid arguments: T2V_ERR_INVALID_ARG. */
int t2v_trace_set(unsigned long long* dev_records, int64_t capacity);
int t2v_trace_count(int64_t* n_records, int* n_overflowed);

/* MFMA throughput probe, for measurement context only (not part of the attention path).
 * Launches `blocks` workgroups of four waves; each wave runs four independent chains of
 * `iters` v_mfma_f32_32x32x16_bf16 with no memory traffic, on `stream`, and waits for it.
 *   rec         device unsigned long long[3 * blocks], caller-owned; per workgroup: shader
 *               clock ticks, wall-clock ticks, a checksum word (overwritten)
 *   blocks      1 .. 2^20;  iters 1 .. 2^24
 *   ms_out      elapsed milliseconds between HIP events around the launch
 *   tflops_out  bf16 dense TFLOP/s achieved (2 * 32 * 32 * 16 flops per MFMA)
 *   ghz_out     average shader clock over the run (clock ticks / wall-clock ticks times the
 *               device's wall-clock rate)
 * NULL pointers or sizes out of range: T2V_ERR_INVALID_ARG before any launch; HIP failures:
 * T2V_ERR_HIP. */
int t2v_probe_mfma_peak(unsigned long long* rec, int blocks, int iters, void* stream, double* ms_out,
                        double* tflops_out, double* ghz_out);

/* Library version, for diagnostics. */
const char* t2v_version(void);

#ifdef __cplusplus
}
#endif

#endif /* T2VATTN_H */
