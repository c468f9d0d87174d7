/*
 * revisit.h -- C interface of librevisit, the GPU (gfx950) hot path of
 * training-free revisit consistency for autoregressive generative rendering
 * (arXiv 2607.21848: pose-retrieved loop-closure memory, Sec. 4.2, and the
 * geometric correspondence attention prior, Sec. 4.3).
 *
 * Three stages, one entry point each, and the cache packing that puts the
 * retrieved chunks in front of the attention:
 *
 *   retrieve_chunks           -- pose retrieval over the history bank
 *                                (Sec. 4.2, Eq. retrieval)
 *   reproject_correspondence  -- per-token depth/pose reprojection into the
 *                                retrieved frames with the occlusion test
 *                                (Sec. 4.3, Eq. reprojection, Eq. visibility)
 *   reproject_rotation        -- the fixed-centre case of the same: the
 *                                rotation / zoom homography, no depth
 *                                (Sec. 4.3)
 *   biased_chunk_attention    -- chunk attention with the Gaussian
 *                                correspondence bias fused in
 *                                (Sec. 4.3, Eq. bias)
 *   pack_retrieved_kv         -- gather of the retrieved chunks' keys and
 *                                values into the cache, keys re-rotated to
 *                                the packed positions (Sec. 4.2)
 *
 * and a streaming driver (rc_stream_*) that runs the paper's cache layout
 * chunk by chunk on the device.
 *
 * Conventions common to all entry points
 * --------------------------------------
 * - Every array argument is a DEVICE pointer owned by the caller and must
 *   stay valid until the work queued on `stream` has completed. Outputs must
 *   not alias inputs. The stage calls allocate nothing and synchronise
 *   nothing: where a kernel needs scratch memory (the key split of the bf16
 *   attention, the segmented retrieval of large banks) the caller passes a
 *   device workspace whose size the matching rc_*_workspace_size() query
 *   returns. The only state kept by the library is a per-thread last-error
 *   string; stream objects (rc_stream_create) own device memory that the
 *   caller holds through the handle.
 * - Calls are asynchronous on `stream` (NULL = the default stream). Work on
 *   one workspace must not overlap in time: two calls that may run
 *   concurrently (different streams) need different workspaces.
 * - Arguments are validated on the host before anything is queued: on a
 *   non-zero status nothing has been enqueued and rc_last_error() says why
 *   (the one exception, rc_stream_step, is stated there).
 *   Device-resident index arrays (slots, selections) cannot be checked from
 *   the host; out-of-range entries there are given a defined meaning below
 *   instead of being read out of bounds.
 * - No C++ exception crosses this interface.
 * - Poses are row-major 4x4 camera-to-world matrices [R | c; 0 0 0 1]
 *   (Sec. 4.1: camera-to-world rotation and centre), camera axes x right,
 *   y down, z forward; planar depth is the camera-frame z (Sec. 4.1).
 * - Intrinsics are (fx, fy, cx, cy) in depth-map pixel units, pixel (x, y)
 *   covering [x, x+1) x [y, y+1). A token is a p x p block of depth pixels;
 *   the token-grid intrinsics of Sec. 4.1 are these divided by p.
 */
#ifndef REVISIT_H
#define REVISIT_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
enum {
    REVISIT_OK = 0,
    REVISIT_ERR_NULL = 1,        /* a required pointer is NULL */
    REVISIT_ERR_SHAPE = 2,       /* a size is negative, inconsistent or too large */
    REVISIT_ERR_UNSUPPORTED = 3, /* dtype / head dimension not built */
    REVISIT_ERR_PARAM = 4,       /* a method parameter is out of its domain */
    REVISIT_ERR_LAUNCH = 5,      /* the HIP runtime refused the launch */
    REVISIT_ERR_MEMORY = 6       /* device or host memory could not be allocated */
};

/* Element types of biased_chunk_attention (and of the other calls where they
 * apply). REVISIT_FP8_QK: q and k in fp8 e4m3 (OCP: 1 sign, 4 exponent bits
 * with bias 7, 3 mantissa bits, no infinities, 0x7f / 0xff NaN), v and o in
 * bf16. */
enum { REVISIT_BF16 = 1, REVISIT_F32 = 2, REVISIT_FP8_QK = 3 };

/* Correspondence reason codes written to out_idx by reproject_correspondence
 * and reproject_rotation (the rejection causes of Sec. 4.3, design choice
 * (iii), plus an empty retrieved slot and, for the rotation-only path, a
 * source whose centre is not the target's). A value >= 0 is a key index
 * within the source frame. */
enum {
    REVISIT_UNDEFINED = -1, /* query depth not finite or <= 0 */
    REVISIT_BEHIND = -2,    /* [X_s]_z <= 0 */
    REVISIT_OFF_GRID = -3,  /* u^ outside [0, w) x [0, h) */
    REVISIT_OCCLUDED = -4,  /* Eq. visibility fails (or source depth NaN) */
    REVISIT_NO_SOURCE = -5, /* the retrieved slot is empty */
    REVISIT_CENTRE_MOVED = -6 /* reproject_rotation only: c_s != c_t */
};

/* Largest k accepted by retrieve_chunks. */
#define REVISIT_MAX_K 32

/* Human-readable name of a status code (static string). */
const char* rc_status_string(int status);

/* Detail of the last non-zero status returned on the calling thread
 * (static per-thread buffer, overwritten by the next failing call). */
const char* rc_last_error(void);

/*
 * retrieve_chunks -- Sec. 4.2, Eq. retrieval.
 *
 * For each query chunk q with pose query_c2w[q] and chunk index
 * n = query_chunk[q], score every bank entry j (entry j IS chunk j):
 *     s(j) = |c_j - c_n| / E + w_v (1 - v_j . v_n)
 * with c = last column of the pose and v = R e_z (third column, used as
 * stored), keep j if j >= first_candidate, n - j >= delta,
 * |c_j - c_n| / E <= tau_c and v_j . v_n >= cos(tau_v), and return the k
 * admissible entries of smallest score, ties broken by smaller j. Scores
 * are evaluated in double precision; cos(tau_v) is evaluated once on the
 * host.
 *
 *   bank_c2w      [n_bank][4][4] fp32   one representative pose per chunk
 *   query_c2w     [n_query][4][4] fp32
 *   query_chunk   [n_query] int32       n of each query
 *   E > 0, w_v, tau_c, tau_v (radians): finite
 *   k             1..REVISIT_MAX_K
 *   out_idx       [n_query][k] int32    chunk ids, -1 past the count
 *   out_score     [n_query][k] fp32     nullable; s rounded to fp32, +inf past the count
 *   out_count     [n_query] int32       number of admissible entries returned (0..k);
 *                                       count < k means the retrieved slot
 *                                       extends the recent window (Sec. 4.2)
 *   frames_per_chunk, out_frame_sel  nullable [n_query][k * frames_per_chunk]:
 *                 entry i*F + f = out_idx[i]*F + f, or -1 past the count; this
 *                 is the source-frame selection reproject_correspondence takes.
 *
 * n_bank == 0 or n_query == 0 is valid (count 0 / nothing to do).
 * n_bank <= 2^30; bank_c2w must be 8-byte aligned (REVISIT_ERR_SHAPE
 * otherwise). Banks of more than 8192 entries are scanned by many waves
 * (workgroups of 16 waves over segments of 16384 entries) whose k best
 * candidates are merged in the same (score, index) order, with the same
 * result; the segments' candidates go to the caller's workspace.
 *
 *   workspace, workspace_bytes  device scratch of at least the size
 *                 rc_retrieve_workspace_size() returns for (n_bank, n_query,
 *                 k), 16-byte aligned; may be NULL / 0 when that size is 0
 *                 (banks of at most 8192 entries). Too small:
 *                 REVISIT_ERR_SHAPE; NULL while needed: REVISIT_ERR_NULL.
 */
int retrieve_chunks(const float* bank_c2w, int32_t n_bank,
                    const float* query_c2w, const int32_t* query_chunk, int32_t n_query,
                    float E, float w_v, float tau_c, float tau_v,
                    int32_t delta, int32_t first_candidate, int32_t k,
                    int32_t* out_idx, float* out_score, int32_t* out_count,
                    int32_t frames_per_chunk, int32_t* out_frame_sel,
                    void* workspace, size_t workspace_bytes,
                    hipStream_t stream);

/*
 * rc_retrieve_workspace_size -- bytes of workspace retrieve_chunks needs for
 * a bank of n_bank entries, n_query queries and k results per query:
 * n_query * segments * k * 12 with segments = ceil(n_bank / 16384) above
 * 8192 entries, else 0. The arguments are validated as by retrieve_chunks.
 */
int rc_retrieve_workspace_size(int32_t n_bank, int32_t n_query, int32_t k, size_t* bytes);

/*
 * reproject_correspondence -- Sec. 4.3, Eq. reprojection and Eq. visibility.
 *
 * For B independent problems, every token p of every target frame t and every
 * source frame s:
 *     z_p  = mean of the token's p x p depth pixels (row-major sum)
 *     X_t  = z_p K_t^-1 u~_p,   u_p = (col + 1/2, row + 1/2) token units
 *     X_s  = R_s^T (R_t X_t + c_t - c_s)
 *     u^   = pi(K_s X_s)
 * accepted iff 0 <= u^_x < w, 0 <= u^_y < h and
 *     [X_s]_z <= (1 + eps) D_s(u^),   D_s = pooled depth of the cell holding u^.
 * All arithmetic is IEEE double in exactly this order (no contraction), so the
 * results are reproducible bit for bit on any IEEE host.
 *
 *   tgt_depth [B][Tq][h*p][w*p] fp32, tgt_c2w [B][Tq][4][4], tgt_K [B][Tq][4]
 *   sources, either
 *     src_sel == NULL: src_depth [B][S][h*p][w*p], src_c2w [B][S][4][4],
 *                      src_K [B][S][4] (n_src ignored), or
 *     src_sel != NULL: a frame bank src_depth [n_src][h*p][w*p], src_c2w
 *                      [n_src][4][4], src_K [n_src][4] shared by all problems,
 *                      and src_sel [B][S] int32 choosing the frame of each slot;
 *                      an entry outside [0, n_src) means "no source" and the
 *                      whole slot is written as REVISIT_NO_SOURCE.
 *   S <= 64 source frames per problem; p >= 1 latent pixels per token side;
 *   eps >= 0 finite.
 *   out_uv  [B][S][Tq*h*w][2] fp32: u^ in token units (row-major token order,
 *           target frames outer); NaN for UNDEFINED, BEHIND and NO_SOURCE.
 *   out_idx [B][S][Tq*h*w] int32: key index floor(u^_y) w + floor(u^_x) within
 *           the source frame, or a negative REVISIT_* reason code.
 *
 * Any of B, Tq, S equal to 0 is valid (nothing to do). out_uv must be 8-byte
 * aligned (REVISIT_ERR_SHAPE otherwise).
 */
int reproject_correspondence(const float* tgt_depth, const float* tgt_c2w, const float* tgt_K,
                             const float* src_depth, const float* src_c2w, const float* src_K,
                             const int32_t* src_sel, int32_t n_src,
                             int32_t B, int32_t Tq, int32_t S, int32_t h, int32_t w, int32_t p,
                             float eps,
                             float* out_uv, int32_t* out_idx,
                             hipStream_t stream);

/*
 * biased_chunk_attention -- Sec. 4.3, Eq. bias and design choices (ii)-(iii).
 *
 * Per head, with no mask (every query sees all Lk keys):
 *     A_pk = softmax_scale * q_p . k_k + lambda * B_s(p, k)
 *     B_s(p, k) = -|u_k - u^_s(p)|^2 / (2 sigma^2)
 *     O = softmax_k(A) V,   LSE_p = log sum_k exp(A_pk)  (natural log)
 * The bias applies only to key columns of KV frames whose slot is a retrieved
 * frame s in [0, S), and only for queries with corr_idx[s][p] >= 0; every
 * other logit is the plain scaled dot product. u_k = (k_x + 1/2, k_y + 1/2)
 * with (k_y, k_x) = divmod(k mod (h w), w). The bias is computed on the fly
 * from the correspondence map, never materialised.
 *
 *   dtype       REVISIT_BF16 (D = 128), REVISIT_F32 (D = 64 or 128) or
 *               REVISIT_FP8_QK (D = 128: q, k fp8 e4m3, v, o bf16; the
 *               logits come from the fp8 matrix cores, so any dequantisation
 *               scales of q and k belong in softmax_scale)
 *   q           [Lq][H][D], k, v [Lk][H][D], o [Lq][H][D] in dtype
 *               (fp32 accumulation and softmax in every case)
 *   lse         nullable [H][Lq] fp32
 *   Lq >= 0, Lk >= 1, Lk % (h*w) == 0, Lk / (h*w) <= 1024 KV frames
 *   kv_frame_slot [Lk/(h*w)] int32: s in [0, S) for a retrieved frame, any
 *               other value = unbiased (anchor / recent / current frames)
 *   corr_uv     [S][Lq][2] fp32, corr_idx [S][Lq] int32 (reproject_correspondence
 *               output for this chunk's Lq query tokens); S == 0 or
 *               lambda == 0 turns the bias off (pointers may then be NULL)
 *   softmax_scale > 0 (normally 1/sqrt(D)), sigma > 0, lambda finite.
 *   q, k, v, o must be 16-byte aligned and corr_uv 8-byte aligned
 *   (REVISIT_ERR_SHAPE otherwise). With the bias on, the bf16 and fp8 paths
 *   take token grids of at most 256 x 256 (REVISIT_ERR_SHAPE otherwise).
 *
 * Lq == 0 is valid (nothing to do).
 *
 * Bias precision. The fp32 path evaluates each bias term directly,
 * -gamma ((u_k,x - u^_x)^2 + (u_k,y - u^_y)^2) with the differences taken
 * first (gamma = lambda / (2 sigma^2 softmax_scale), in units of q . k), so
 * its error is a few fp32 units of the term itself. The bf16 and fp8 paths add
 * the bias on the matrix cores in separable form, 2 gamma a . u' - gamma |a|^2
 * - gamma |u'|^2 with a, u' the key and query positions relative to the grid
 * centre, each factor split exactly into bf16 pieces and summed in fp32: their
 * absolute logit error is a few fp32 units (2^-24 relative) of
 * lambda (|a|^2 + |u'|^2) / (2 sigma^2), which for in-grid u^ is at most
 * lambda (h^2 + w^2) / (4 sigma^2): one unit is 1.3e-5 at sigma = 2 on a
 * 30 x 52 grid and 8e-3 at sigma = 0.5 on 256 x 256.
 *
 * bf16 work split: each (head, 128-query tile) item runs on one workgroup,
 * or its keys are cut into P equal parts that run on P workgroups, and a
 * second kernel on the same stream merges the parts from fp32 partial
 * results kept in the workspace.
 *   key_parts   0 = P chosen from the shape and the compute units of the
 *               current device (more parts when the items alone would leave
 *               part of the GPU idle in the last round of workgroups), or a
 *               fixed P in [1, 64] (clamped to the number of 32-key tiles).
 *               Any P gives the same result up to the fp32 rounding of the
 *               merge. fp32 ignores it.
 *   workspace, workspace_bytes  device scratch of at least the size
 *               rc_attention_workspace_size() returns for the same dtype,
 *               shape and key_parts on the same device (items * P * 66.5 KiB
 *               when P > 1, else 0), 16-byte aligned; may be NULL / 0 when
 *               that size is 0. Too small: REVISIT_ERR_SHAPE; NULL while
 *               needed: REVISIT_ERR_NULL.
 */
int biased_chunk_attention(const void* q, const void* k, const void* v, void* o,
                           float* lse, int32_t dtype,
                           int32_t Lq, int32_t Lk, int32_t H, int32_t D, int32_t h, int32_t w,
                           const int32_t* kv_frame_slot,
                           const float* corr_uv, const int32_t* corr_idx, int32_t S,
                           float softmax_scale, float lambda, float sigma,
                           int32_t key_parts, void* workspace, size_t workspace_bytes,
                           hipStream_t stream);

/*
 * rc_attention_workspace_size -- bytes of workspace biased_chunk_attention
 * needs for this dtype, shape and key_parts on the current device (the
 * automatic key_parts = 0 depends on its compute units). Shape and dtype are
 * validated as by biased_chunk_attention.
 */
int rc_attention_workspace_size(int32_t dtype, int32_t Lq, int32_t Lk, int32_t H, int32_t D,
                                int32_t key_parts, size_t* bytes);

/*
 * biased_chunk_attention_noalloc -- for callers that cannot allocate device
 * memory or bring a workspace (code under HIP graph capture without one,
 * tight serving loops, harnesses that forbid allocation): the same
 * arguments, validation and results as biased_chunk_attention, minus the
 * workspace. It allocates nothing. The bf16 / fp8 key split keeps its
 * partial results in a library array of 128 MiB per device (a static device
 * array: each device the library runs on holds its own copy until the
 * process ends).
 *   key_parts = 0  the automatic split, cut to the most parts whose partial
 *                  results fit in 128 MiB (items * P * 66.5 KiB); the results
 *                  then equal biased_chunk_attention's with that P;
 *   key_parts > 0  as for biased_chunk_attention; REVISIT_ERR_SHAPE when its
 *                  partial results need more than 128 MiB.
 * Every call on one device shares that device's array, which keeps the last
 * call's contents: calls that may overlap in time on one device (different
 * streams, graph replays beside other calls) race, and the caller must
 * order them. Nothing in it needs to start at zero: every partial result the
 * merge reads is written earlier in the same call. The first call on a
 * device looks the array's address up (REVISIT_ERR_LAUNCH if that fails).
 */
int biased_chunk_attention_noalloc(const void* q, const void* k, const void* v, void* o,
                                   float* lse, int32_t dtype,
                                   int32_t Lq, int32_t Lk, int32_t H, int32_t D, int32_t h, int32_t w,
                                   const int32_t* kv_frame_slot,
                                   const float* corr_uv, const int32_t* corr_idx, int32_t S,
                                   float softmax_scale, float lambda, float sigma,
                                   int32_t key_parts, hipStream_t stream);

/*
 * pack_retrieved_kv -- Sec. 4.2, cache layout and cache packing.
 *
 * Reinstates retrieved chunks into the attention cache. The history store
 * keeps every historical chunk's keys and values as the cache held them, keys
 * carrying the rotary position embedding of temporal position pos[j] + f in
 * frame f of chunk j. For every layer l and slot s with j = sel[s] in
 * [0, n_store), and T = F h w tokens per chunk:
 *     V_cache[l][dst_row0 + s T + r] = V_store[l][j][r]
 *     K_cache[l][dst_row0 + s T + r] = K_store[l][j][r] with each temporal
 *         pair (k_{2i}, k_{2i+1}), i < rope_t_pairs, read as k_{2i} + i k_{2i+1}
 *         and multiplied by exp(i delta omega_i),
 *         omega_i = rope_theta^(-i / rope_t_pairs),
 *         delta = dst_pos + s F - pos[j]
 * so slot s sits at frame positions dst_pos + s F .. dst_pos + s F + F - 1;
 * the caller chooses dst_pos so that the slots end where the recent window
 * begins (the paper places the retrieved chunk directly next to it). Pairs
 * i >= rope_t_pairs (the grid row and column bands of the embedding) and all
 * values are copied bit for bit. The rotation is evaluated in double
 * precision (x c - y s, x s + y c) and rounded once to the storage type,
 * to nearest even.
 *
 *   dtype         REVISIT_BF16 or REVISIT_F32; D a multiple of 8 in [8, 512]
 *   store_k, store_v  [n_layers][n_store][T][H][D]   (chunk j at index j)
 *   store_pos     nullable [n_store] int32: stored frame position of frame 0 of
 *                 chunk j; NULL means F j (the chunk's original index)
 *   sel           [n_sel] int32: chunk of each slot (e.g. out_idx of
 *                 retrieve_chunks for one query); an entry outside
 *                 [0, n_store) leaves that slot of the cache untouched (the
 *                 caller fills it, e.g. with the recent-window extension
 *                 when no chunk was admissible)
 *   cache_k, cache_v  [n_layers][cache_rows][H][D]; the slots occupy rows
 *                 [dst_row0, dst_row0 + n_sel T), which must fit in cache_rows
 *   rope_t_pairs  temporal pairs, 0..D/2 (0 = plain gather); rope_theta > 0
 *
 * Store and cache must not overlap. store_k, store_v, cache_k, cache_v must be
 * 16-byte aligned, sel and store_pos 4-byte aligned (REVISIT_ERR_SHAPE
 * otherwise). n_layers == 0 or n_sel == 0 is valid (nothing to do); with
 * n_store == 0 every slot is left untouched and the store pointers may be NULL.
 */
int pack_retrieved_kv(const void* store_k, const void* store_v,
                      const int32_t* store_pos, int32_t n_store,
                      const int32_t* sel, int32_t n_sel, int32_t dst_pos,
                      void* cache_k, void* cache_v, int32_t dst_row0, int32_t cache_rows,
                      int32_t n_layers, int32_t dtype,
                      int32_t F, int32_t h, int32_t w, int32_t H, int32_t D,
                      int32_t rope_t_pairs, float rope_theta,
                      hipStream_t stream);

/*
 * reproject_rotation -- Sec. 4.3, the fixed-centre case of Eq. reprojection.
 *
 * For sources that share the target's camera centre (c_s = c_t) the depth
 * scales X_s and cancels under pi, so u^ = pi(K_s R_s^T R_t K_t^-1 u~) is a
 * homography per (target, source) frame pair, independent of depth. This
 * entry point evaluates it without reading any depth: the visibility test of
 * Eq. visibility is not applied (one centre means no parallax and so no
 * disocclusion), and REVISIT_UNDEFINED and REVISIT_OCCLUDED never occur.
 * Per pair, in double:
 *     A = R_s^T R_t,  A[r][c] = (Rs[0][r] Rt[0][c] + Rs[1][r] Rt[1][c]) + Rs[2][r] Rt[2][c]
 *     M = K_s A,      rows (fx_s A0 + cx_s A2, fy_s A1 + cy_s A2, A2)
 *     H = M K_t^-1,   H[r] = (M[r][0] / fx_t, M[r][1] / fy_t,
 *                             (M[r][2] - H[r][0] cx_t) - H[r][1] cy_t)
 * (token-grid intrinsics, i.e. divided by p), then per token
 *     v = H (u_x, u_y, 1),  REVISIT_BEHIND iff v_z <= 0,  u^ = (v_x / v_z, v_y / v_z)
 * with the grid test and key index of reproject_correspondence; no
 * contraction, so the results are reproducible bit for bit. A pair whose fp32
 * centres (the last pose column) are not equal is written as
 * REVISIT_CENTRE_MOVED for every token, u^ NaN.
 *
 *   tgt_c2w [B][Tq][4][4], tgt_K [B][Tq][4] fp32;
 *   sources src_c2w, src_K ([B][S][..], or a frame bank [n_src][..] chosen by
 *   src_sel [B][S]) exactly as for reproject_correspondence;
 *   h, w token grid; p >= 1 latent pixels per token side (intrinsics are in
 *   depth-map pixels, as everywhere);
 *   out_uv [B][S][Tq*h*w][2] fp32 (NaN for BEHIND, NO_SOURCE, CENTRE_MOVED),
 *   out_idx [B][S][Tq*h*w] int32.
 * Any of B, Tq, S equal to 0 is valid (nothing to do); S <= 64; out_uv must
 * be 8-byte aligned (REVISIT_ERR_SHAPE otherwise).
 */
int reproject_rotation(const float* tgt_c2w, const float* tgt_K, const float* src_c2w, const float* src_K,
                       const int32_t* src_sel, int32_t n_src, int32_t B, int32_t Tq, int32_t S,
                       int32_t h, int32_t w, int32_t p, float* out_uv, int32_t* out_idx,
                       hipStream_t stream);

/*
 * pool_token_depth -- the query and source depth of Sec. 4.3 at token
 * resolution (z_p = D_t(u_p) read per token), computed once per stored frame.
 *
 * out[f][r][c] = mean of the p x p block of depth pixels of token (r, c) of
 * frame f, summed row-major (block row outer) in double and rounded to fp32
 * once. Feeding pooled maps to reproject_correspondence with p = 1 and
 * intrinsics divided by p reads 4 bytes of target depth per token instead of
 * 4 p^2; where a block's mean is exact in fp32 the result is bit-identical to
 * the full-resolution call.
 *
 *   depth [n_frames][h p][w p] fp32, out [n_frames][h][w] fp32 (4-byte aligned)
 * n_frames == 0 is valid (nothing to do).
 */
int pool_token_depth(const float* depth, int32_t n_frames, int32_t h, int32_t w, int32_t p,
                     float* out, hipStream_t stream);

/*
 * Streaming driver -- Sec. 4.2 (cache layout, loop-closure retrieval, cache
 * packing) and Sec. 4.3, run chunk by chunk over one generated sequence.
 *
 * A stream object owns the device memory of the sequence: the pose bank
 * (max_chunks poses), the history ring and the packed attention cache. The
 * ring keeps the anchor and the capacity - 1 newest chunks: per chunk the
 * pre-pooled token depth, the frame poses, the token-grid intrinsics (K / p)
 * and every layer's keys and values. Chunk m >= 1 lives at ring slot
 * 1 + (m - 1) mod (capacity - 1). rc_stream_step() runs chunk n = 0, 1, 2, ...
 * and enqueues everything on `stream` without host synchronisation:
 *   1. the chunk enters the ring (depth pooled to the token grid: p x p mean
 *      in double rounded to fp32) and its middle frame's pose the bank;
 *   2. retrieval (Eq. retrieval, k = 1) over the resident chunks 1..n-1,
 *      i.e. first candidate max(1, n - capacity + 2);
 *   3. the layout of the attention range, in this order and with these frame
 *      positions: anchor chunk 0 (0..F-1), the retrieved chunk (F..2F-1) --
 *      or, when nothing is admissible, chunk n-3 as the extension of the
 *      recent window, unbiased --, recent chunks n-2 (2F..) and n-1 (3F..),
 *      and the current chunk (4F..5F-1); parts that do not exist yet are
 *      left out (the retrieved slot exists from n = 4 on). The retrieved
 *      part's ring slot, the KV frame slot table and the source frames of
 *      step 4 are built on the device from the retrieval result;
 *   4. correspondence (Eq. reprojection, Eq. visibility) of the chunk's tokens
 *      into the retrieved chunk's F frames, on the pooled maps (p = 1);
 *   5. the packed cache of every layer (pack_retrieved_kv; keys enter the
 *      ring with the embedding of position 4F + f, as the network produced
 *      them for the current role, and are re-rotated to their role's
 *      position); the anchor's rows, the same from chunk 1 on, are packed
 *      at chunk 1 only;
 *   6. biased attention (Eq. bias) of every layer over its packed cache,
 *      the retrieved frames carrying slots 0..F-1 when a chunk was retrieved.
 *
 * rc_stream_create -- allocates the stream on the current device.
 *   dtype REVISIT_BF16 (D = 128, h, w <= 256) or REVISIT_F32 (D = 64 or 128); 1 <= F <= 64;
 *   capacity >= 5 (keeps chunk n-3 resident); method parameters as for the
 *   stage entry points. Allocation failure: REVISIT_ERR_MEMORY, nothing kept.
 *   Device memory: layers * capacity * F h w * H * D * 2 (K and V) elements
 *   for the ring plus layers * 5 F h w * H * D * 2 for the cache, plus small
 *   tables.
 *   The object also owns the attention key-split and retrieval workspace of
 *   its largest step, sized here for the current device.
 * rc_stream_step -- runs the next chunk. Inputs (device, caller-owned):
 *   depth [F][h p][w p] fp32 planar depth, c2w [F][4][4], K [F][4] depth-pixel
 *   intrinsics; q, k, v [layers][F h w][H][D] in dtype (k with the rotary
 *   embedding of positions 4F + f); outputs o [layers][F h w][H][D] and lse
 *   (nullable) [layers][H][F h w]. The device must be the one the stream was
 *   created on. Steps of one stream must be issued in order on one stream
 *   (they share the object's buffers); REVISIT_ERR_SHAPE once max_chunks
 *   chunks have run. Every argument and the whole step's configuration are
 *   validated before the first launch, so a status other than
 *   REVISIT_ERR_LAUNCH means nothing was enqueued. The exception: when the
 *   HIP runtime refuses one of the step's launches (REVISIT_ERR_LAUNCH), the
 *   stages before it stay queued and the step does not advance; issuing
 *   the same chunk again redoes them (each writes the same ring slot and
 *   tables).
 * rc_stream_view -- device pointers to the last step's intermediate results
 *   (retrieval, layout tables, correspondence, packed cache) and its layout
 *   sizes, for inspection; valid until the next step or rc_stream_destroy.
 * rc_stream_destroy -- waits for the device and frees everything (NULL: no-op).
 */
typedef struct rc_stream rc_stream;

typedef struct {
    int32_t F, h, w, p;           /* frames per chunk, token grid, depth pixels per token side */
    int32_t H, D, layers, dtype;  /* heads, head dim, transformer layers, REVISIT_BF16 / REVISIT_F32 */
    int32_t capacity;             /* history ring chunks, >= 5 */
    int32_t max_chunks;           /* pose bank length: chunks the stream may run */
    float E, w_v, tau_c, tau_v;   /* retrieval (Eq. retrieval), tau_v in radians */
    int32_t delta;                /* temporal gap gate */
    float eps, lambda, sigma, softmax_scale;  /* visibility tolerance and bias (Sec. 4.3) */
    int32_t rope_t_pairs;         /* temporal pairs of the rotary embedding (0..D/2) */
    float rope_theta;
} rc_stream_config;

typedef struct {
    int32_t n;          /* chunk id of the last step, -1 before the first */
    int32_t n_parts;    /* parts of its attention range, in layout order */
    int32_t ret_part;   /* index of the retrieved / extension part, -1 if absent */
    int32_t Lk;         /* keys per layer: n_parts F h w */
    int32_t cache_rows; /* rows per layer of the cache arrays: 5 F h w */
    const int32_t* ret_idx;    /* [1] retrieved chunk or -1 (n >= 1) */
    const int32_t* ret_count;  /* [1] 0 or 1 (n >= 1) */
    const int32_t* part_slot;  /* [n_parts] ring slot of every part */
    const int32_t* kv_slot;    /* [n_parts F] KV frame slot table */
    const int32_t* src_sel;    /* [F] ring frames of the retrieved chunk, or -1 */
    const float* corr_uv;      /* [F][F h w][2] (ret_part >= 0) */
    const int32_t* corr_idx;   /* [F][F h w]    (ret_part >= 0) */
    const void* cache_k;       /* [layers][cache_rows][H][D], first Lk rows valid */
    const void* cache_v;
} rc_stream_state;

int rc_stream_create(const rc_stream_config* cfg, rc_stream** out);
int rc_stream_step(rc_stream* s, const float* depth, const float* c2w, const float* K,
                   const void* q, const void* k, const void* v, void* o, float* lse,
                   hipStream_t stream);
int rc_stream_view(const rc_stream* s, rc_stream_state* out);
int rc_stream_destroy(rc_stream* s);

#ifdef __cplusplus
}
#endif

#endif /* REVISIT_H */
