/*
 * libbifattn -- bifurcated incremental-decoding attention on AMD MI355X (gfx950).
 *
 * Method (Bifurcated Attention, Section 4.2, Eq. 3 and Eq. 4): for b samples
 * that share one prefill context, the attention of each new query token is
 * split along the key axis into a context part, which reads ONE copy of the
 * context cache K_c/V_c for all samples, and a decode part, which reads each
 * sample's own cache K_d/V_d. One softmax spans both parts, so the result is
 * exactly standard multi-group attention (Section 3.3, Eq. 1-2; proof in
 * Appendix E.1) while the KV bytes read drop from g*k*b*(m_c+m_d) to
 * g*k*(m_c + b*m_d) (Section 4.3).
 *
 * Notation (Section 3.1): b samples, h query heads, g KV groups with
 * p = h/g query heads per group (g = h: multi-head, g = 1: multi-query),
 * d head dimension (the paper's k), m_c context length, m_d_max capacity of
 * each sample's decode cache, len_i <= m_d_max its valid rows, n new tokens
 * per sample: 1 in incremental decoding, n_g > 1 when draft tokens are
 * verified in one step (the appendix on speculative decoding, where n_g
 * replaces the query length n of Eq. 3-4).
 *
 * Layouts (all row-major, all device memory, bf16 = 16-bit brain float):
 *   q       bf16 [b][h][n][d]       token r of head j of sample i at ((i*h + j)*n + r)*d
 *                                   ([b][h][d] when n = 1)
 *   Kc, Vc  kv  [g][m_c][d]         one shared copy of the context cache
 *   Kd, Vd  kv  [b][g][m_d_max][d]  per-sample decode cache (int4: d/2 bytes a row)
 *   decode_lens int32 [b]           valid decode rows per sample
 *   k_scale, v_scale fp32 [g]       per-group key / value scales (optional)
 *   out     fp32 [b][h][n][d]
 * kv is the plan's cache element type (dims.kv_type): bf16, 8-bit codes
 * (OCP fp8 E4M3, or two's complement int8), one byte each, or two's
 * complement int4 codes, two per byte. The FAQ on attention quantization
 * notes that 8-bit KV halves the KV bytes (4-bit KV quarters them) and leaves
 * the method unchanged; here the key of a cache row is k_scale[gam] times
 * its codes' values and its value v_scale[gam] times its codes' values, the
 * same scales for the group's context and decode caches (NULL scales mean
 * 1). Codes are widened to bf16 exactly; the scales enter in fp32.
 * Head j reads KV group j / p (group-major, the bgpnk order of Eq. 1).
 * Decode rows t >= len_i are never read into arithmetic: they may hold
 * anything, NaN included. With n > 1 the n new tokens are the last n of the
 * len_i valid decode rows, and token r attends to the context and to decode
 * rows t < len_i - n + r + 1 (the rows up to and including itself); rows it
 * does not see get weight 0 (they must be finite, like all valid rows). Arithmetic: bf16 products, fp32 logits, softmax
 * statistics and accumulators; softmax weights enter the weighted sum over
 * values rounded to bf16. Softmax scale: dims.scale, or 1/sqrt(d) when 0.
 *
 * Ownership and concurrency: the caller owns every tensor and the stream;
 * the library never frees caller memory. A plan owns its workspace (allocated
 * at create, freed at destroy) on the device current at create; its calls
 * take that device's memory and streams. Calls are asynchronous on the given stream
 * (no host synchronisation) except bifattn_plan_status and
 * bifattn_plan_read_timing. One plan must not be used by two calls that may
 * run concurrently (they share the workspace). Results are bitwise
 * deterministic for a given plan (fixed split counts and merge order, no
 * floating-point atomics).
 *
 * Errors: every entry point returns a bifattn_status_t. Argument errors are
 * detected on the host before anything is enqueued and leave `out`
 * untouched. decode_lens lives on the device, so it is checked there: values
 * outside [0, m_d_max] are clamped into that range and raise a sticky flag
 * that bifattn_plan_status reports as BIFATTN_ELENS.
 */
#ifndef BIFATTN_H
#define BIFATTN_H

#include <stddef.h>
#include <stdint.h>

#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

#define BIFATTN_VERSION 4

typedef enum {
  BIFATTN_OK = 0,
  BIFATTN_EINVAL = -1,       /* null pointer, non-positive size, h % g != 0, ... */
  BIFATTN_EUNSUPPORTED = -2, /* valid but not built: d not in {64,128}, p*n > 64,
                                (m_c + m_d_max) * d * 2 > 2^31 - 1 */
  BIFATTN_EALIGN = -3,       /* a tensor pointer not 16-byte aligned */
  BIFATTN_ENOMEM = -4,       /* workspace or event allocation failed */
  BIFATTN_EHIP = -5,         /* a HIP runtime call or kernel launch failed */
  BIFATTN_ELENS = -6,        /* a decode length was outside [0, m_d_max] */
  BIFATTN_ESCALE = -7,       /* a key or value scale was not a positive normal float */
  BIFATTN_ESCRATCH = -8      /* bifattn_decode_noalloc: workspace beyond its fixed scratch */
} bifattn_status_t;

/* Which computation bifattn_decode runs (bifattn_dims_t.path). The FAQ on
 * caveats notes that splitting the attention in two costs parallelism on
 * small workloads and that a switch on the workload keeps the better of the
 * two: AUTO picks per plan from the shape (see bifattn_plan_create). */
typedef enum {
  BIFATTN_PATH_AUTO = 0,
  BIFATTN_PATH_BIFURCATED = 1, /* context and decode parts, then the combine (Eq. 3-4) */
  BIFATTN_PATH_STANDARD = 2    /* one work-group per (sample, group) over context then
                                  decode rows, output written directly (Eq. 1-2) */
} bifattn_path_t;

/* Cache element types (bifattn_dims_t.kv_type). */
typedef enum {
  BIFATTN_KV_BF16 = 0,     /* bf16 keys and values */
  BIFATTN_KV_FP8_E4M3 = 1, /* OCP 8-bit float E4M3 codes (bias 7, no infinities, max 448) */
  BIFATTN_KV_INT8 = 2,     /* two's complement 8-bit integer codes */
  BIFATTN_KV_INT4 = 3      /* two's complement 4-bit integer codes, two per byte: element u
                              of a row in byte u/2, even u in the low nibble; rows d/2 bytes */
} bifattn_kv_type_t;

/* Problem dimensions (Section 3.1 notation; d is the head dimension). */
typedef struct {
  int32_t b;       /* samples sharing the context, >= 1 */
  int32_t h;       /* query heads, >= 1 */
  int32_t g;       /* KV groups, >= 1, divides h */
  int32_t d;       /* head dimension: 64 or 128 */
  int32_t m_c;     /* context length, >= 1 */
  int32_t m_d_max; /* decode cache capacity per sample, >= 0 */
  float scale;     /* softmax scale on q.k; 0 selects 1/sqrt(d) */
  int32_t n;       /* new tokens per sample, >= 1 (0 is taken as 1) */
  int32_t kv_type; /* a bifattn_kv_type_t: element type of Kc, Vc, Kd, Vd */
  int32_t path;    /* a bifattn_path_t; 0 = choose from the workload */
} bifattn_dims_t;

typedef struct bifattn_plan_s *bifattn_plan_t;

/* How a plan splits the work (read-only, for callers that report it). */
typedef struct {
  int32_t ctx_keys_per_block; /* context keys one work-group reads */
  int32_t ctx_splits;         /* S_c: context partial results per output row */
  int32_t ctx_row_blocks;     /* work-groups sharing one context key chunk */
  int32_t ctx_blocks;         /* context work-groups per call */
  int32_t dec_keys_per_block; /* decode keys one work-group reads */
  int32_t dec_splits;         /* decode partial results per output row */
  int32_t dec_blocks;         /* decode work-groups per call */
  int32_t fused;              /* 1: context and decode parts in one launch */
  int32_t path;               /* the path bifattn_decode runs: BIFATTN_PATH_BIFURCATED or
                                 BIFATTN_PATH_STANDARD */
  size_t workspace_bytes;     /* device memory the plan owns */
  int32_t ctx_kernel;         /* context work-groups: 0 in the partial launch (few rows per
                                 group, or none), 1 many-row kernel of 16-row waves, 2 many-row
                                 32x32 MFMA kernel of 32-row waves */
  int32_t side_stream;        /* 1 when the decode launch runs on the plan's side stream */
} bifattn_plan_info_t;

/* Kernels a plan launches; used to select what bifattn_plan_set_timing times. */
typedef enum {
  BIFATTN_KERNEL_PARTIALS = 0, /* context + decode partial kernel(s) of a call */
  BIFATTN_KERNEL_COMBINE = 1,  /* online-softmax combine of a call */
  BIFATTN_KERNEL_CALL = 2,     /* the whole call, first launch to last */
  BIFATTN_KERNEL_CONTEXT = 3,  /* the launch holding the context work-groups */
  BIFATTN_KERNEL_DECODE = 4    /* the launch holding the decode work-groups */
} bifattn_kernel_t;

/*
 * Validate dims and allocate the plan and its workspace on the current HIP
 * device. On success *plan is set; on failure *plan is left NULL.
 * With dims.path = BIFATTN_PATH_AUTO the plan runs the standard path when
 * every (sample, group) unit fits in one round of work-groups on the GPU
 * (b*g <= 512), a unit has at most 32 query rows ((h/g)*n <= 32) and holds
 * few keys: m_c + m_d_max <= 1100 (<= 600 when b*g > 256), or <= 2200 when
 * b*(h/g)*n >= 64. There one launch without partials beats reading the
 * context once; otherwise the bifurcated path. Both give the same attention
 * (Appendix E.1).
 * Errors: EINVAL (null argument, b/h/g/m_c < 1, m_d_max < 0, n < 0,
 * h % g != 0, unknown kv_type or path, sizes whose byte counts overflow),
 * EUNSUPPORTED (d not 64 or 128, (h/g)*n > 64, or one sample's cache rows
 * (m_c + m_d_max) * d * (bytes per element) beyond 2^31 - 1), ENOMEM
 * (device allocation failed), EHIP (no usable device).
 */
bifattn_status_t bifattn_plan_create(const bifattn_dims_t *dims, bifattn_plan_t *plan);

/* Free the plan and its workspace after waiting for the plan's own device
 * work: the end of its last call (an event every call records on its stream
 * after its last launch) and the plan's own stream. The workspace comes from
 * the stream-ordered allocator and is freed in the plan's stream order, so
 * other streams on the device are not waited for (where that allocator is
 * unavailable the plan falls back to hipMalloc, whose free synchronises the
 * device). NULL is accepted and ignored. */
bifattn_status_t bifattn_plan_destroy(bifattn_plan_t plan);

/* Fill *info with the plan's split decisions. EINVAL on null arguments. */
bifattn_status_t bifattn_plan_get_info(bifattn_plan_t plan, bifattn_plan_info_t *info);

/*
 * One bifurcated decode-attention step (Section 4.2, Eq. 3-4):
 *   out[i, j, r, :] = softmax_t( scale * q[i,j,r,:] . K_i[t,:] ) @ V_i
 * with K_i = Kc[j/p] (+) Kd[i, j/p, 0:len_i - n + r + 1] and V_i likewise. Enqueues on
 * `stream` (a) context partials: each work-group stages a chunk of Kc/Vc of
 * one group once and applies it to all b*p query rows of the group; (b)
 * decode partials: per sample and group over its own Kd/Vd; (c) the combine,
 * which merges the (max, sum, weighted-value) partials of both parts into
 * `out`. With many query rows per group (b*(h/g)*n > 64) and a decode cache
 * of 16 MiB or more, (b) runs on a stream the plan owns, beside (a), and
 * `stream` waits for it before (c). On a plan whose path is BIFATTN_PATH_STANDARD it enqueues one
 * launch instead: per (sample, group), the context rows then the decode
 * rows in one softmax, written to `out`. Kd, Vd and decode_lens may be NULL only when m_d_max == 0.
 * All tensors live on the plan's device (the one current at plan creation)
 * and `stream` belongs to it (NULL: the null stream of the current device,
 * which must then be the plan's).
 * Errors: EINVAL (null plan or required pointer, a stream of another
 * device), EALIGN (q, Kc, Vc, Kd, Vd or out not 16-byte aligned, decode_lens
 * not 4-byte aligned), EHIP (launch failure). Device-side length errors: see
 * bifattn_plan_status.
 */
bifattn_status_t bifattn_decode(bifattn_plan_t plan, const void *q, const void *Kc,
                                const void *Vc, const void *Kd, const void *Vd,
                                const int32_t *decode_lens, float *out, hipStream_t stream);

/*
 * bifattn_decode with per-group scales (the FAQ on attention quantization):
 * keys of group gam are k_scale[gam] times the cache entries, values
 * v_scale[gam] times them, for the context and the decode cache alike. The
 * key scale folds into the softmax scale of the group's work-groups and the
 * value scale into the combine, so the cost is that of bifattn_decode.
 * k_scale, v_scale: device fp32 [g], or NULL for all 1. Scales must be
 * positive normal floats; a call that finds another value sets the plan's
 * device-side flag that bifattn_plan_status reports as BIFATTN_ESCALE, and
 * the output rows of that group are unspecified (NaN possible).
 * Errors: those of bifattn_decode; EALIGN also for a scale pointer that is
 * not 4-byte aligned.
 */
bifattn_status_t bifattn_decode_scaled(bifattn_plan_t plan, const void *q, const void *Kc,
                                       const void *Vc, const void *Kd, const void *Vd,
                                       const int32_t *decode_lens, const float *k_scale,
                                       const float *v_scale, float *out, hipStream_t stream);

/*
 * Ablation without bifurcation (the baseline of Section 4.1): the same
 * attention, but every sample reads its own physically replicated cache
 *   K, V   kv [b][g][m_c + m_d_max][d], rows 0..m_c-1 the context copy,
 *          rows m_c..m_c+len_i-1 the sample's decode rows,
 * so the context is read b times. Same partial and combine kernels, no
 * context part. Same errors as bifattn_decode.
 */
bifattn_status_t bifattn_decode_replicated(bifattn_plan_t plan, const void *q, const void *K,
                                           const void *V, const int32_t *decode_lens,
                                           float *out, hipStream_t stream);

/* The replicated ablation with per-group scales, as bifattn_decode_scaled. */
bifattn_status_t bifattn_decode_replicated_scaled(bifattn_plan_t plan, const void *q,
                                                  const void *K, const void *V,
                                                  const int32_t *decode_lens,
                                                  const float *k_scale, const float *v_scale,
                                                  float *out, hipStream_t stream);

/*
 * Append one decoding step's keys and values to the decode cache (the decode
 * cache holds the keys and values of the previous decoding steps, Section
 * 3.1), so that a generation loop runs append then decode each step:
 *   Kd[i, gam, len_i + r, :] = k_new[i, gam, r, :]   (r < n; Vd likewise)
 *   decode_lens[i] += n
 * k_new, v_new [b][g][n][d] of the plan's cache element type (the step's n
 * new tokens per sample, n from the plan; 8-bit codes, and int4 bytes of
 * two codes, are copied as they are, encoded by the caller with the group's
 * scales); Kd, Vd, decode_lens
 * as in bifattn_decode, updated in place on
 * `stream`. Rows that would pass m_d_max are dropped (the length stops at
 * m_d_max), a length outside [0, m_d_max] is clamped first; both raise the
 * device-side flag that bifattn_plan_status reports as BIFATTN_ELENS.
 * Errors: EINVAL (null argument, m_d_max = 0, a stream of another device
 * than the plan's), EALIGN (a tensor not 16-byte aligned, decode_lens not
 * 4-byte aligned), EHIP (launch failure).
 */
bifattn_status_t bifattn_append_kv(bifattn_plan_t plan, const void *k_new, const void *v_new,
                                   void *Kd, void *Vd, int32_t *decode_lens, hipStream_t stream);

/*
 * Synchronise `stream`, then report and clear the plan's device-side flags:
 * BIFATTN_ESCALE if any call since the last check saw a scale that is not a
 * positive normal float, else BIFATTN_ELENS if one saw a decode length
 * outside [0, m_d_max] (the call used the clamped length) or an append ran
 * out of capacity, else BIFATTN_OK.
 * EHIP if the stream reports an error.
 */
bifattn_status_t bifattn_plan_status(bifattn_plan_t plan, hipStream_t stream);

/*
 * Time the selected kernel of the next `capacity` calls with HIP events
 * (capacity 0 switches timing off). For BIFATTN_KERNEL_PARTIALS and
 * BIFATTN_KERNEL_COMBINE the launches record the events themselves
 * (hipExtLaunchKernel), so they span the kernels' own execution, from the
 * start of the first launch of the section to the end of its last (where a
 * plan runs its decode launch on a side stream beside the many-row context
 * kernel, the partial section is recorded on the call's stream from before
 * the fork to after the join); BIFATTN_KERNEL_CONTEXT and
 * BIFATTN_KERNEL_DECODE time the launch that holds the context (decode)
 * work-groups alone, which is the partial launch itself where one launch
 * holds both (and nothing on the standard path or the replicated ablation); for
 * BIFATTN_KERNEL_CALL they are recorded on the stream around the whole
 * call. Timing stops recording when full. Before replacing the recorder it
 * waits for the plan's own last call (not for the whole device).
 * Errors: EINVAL (bad kernel id or negative capacity), ENOMEM, EHIP.
 */
bifattn_status_t bifattn_plan_set_timing(bifattn_plan_t plan, bifattn_kernel_t kernel,
                                         int32_t capacity);

/*
 * Wait for the recorded events and return the number of timed calls and the
 * sum of their durations in milliseconds; then rewind the recorder.
 */
bifattn_status_t bifattn_plan_read_timing(bifattn_plan_t plan, int32_t *calls, double *total_ms);

/*
 * bifattn_decode_scaled for callers that cannot allocate device memory:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation. It takes the dimensions instead of a plan (creating a plan
 * allocates), computes the same work split on the host (the decode launch
 * always on `stream`, never on a side stream), and keeps its partials and
 * status word in a fixed scratch buffer of BIFATTN_NOALLOC_SCRATCH_BYTES
 * (64 MiB) that the library holds on each GPU from its load to the end of
 * the process. It calls no allocator, creates no stream or event, and
 * enqueues only kernel launches on `stream`. Arguments, layouts, scale and
 * length handling are those of bifattn_decode_scaled.
 * Every call on one GPU shares that GPU's scratch buffer, which keeps the
 * last call's partials: calls that may overlap on one GPU (two streams, or
 * one stream and a graph replay) race on it and must be serialised by the
 * caller. Device-side checks still clamp out-of-range lengths, but their
 * flags are not reported (there is no plan to query).
 * Errors: those of bifattn_plan_create's validation and of
 * bifattn_decode_scaled's argument checks; BIFATTN_ESCRATCH (nothing is
 * enqueued) when the problem's workspace exceeds the scratch buffer: it
 * holds g*S_c*b*(h/g)*n context partials and b*g*S_d*4*(h/g)*n decode
 * partials of (d + 2)*4 bytes each (S_c context splits and S_d decode
 * chunks of the work split without a side stream), about 4.3 MB for the
 * 32-sample 7B-shaped MHA layer and 51 MB for the 256-sample GQA layer over
 * a 32k context. The size check comes before any HIP call.
 */
#define BIFATTN_NOALLOC_SCRATCH_BYTES (64u << 20)
bifattn_status_t bifattn_decode_noalloc(const bifattn_dims_t *dims, const void *q, const void *Kc,
                                        const void *Vc, const void *Kd, const void *Vd,
                                        const int32_t *decode_lens, const float *k_scale,
                                        const float *v_scale, float *out, hipStream_t stream);

/* Static text for a status code. Never NULL. */
const char *bifattn_status_string(bifattn_status_t status);

/* BIFATTN_VERSION of the built library. */
int32_t bifattn_version(void);

#ifdef __cplusplus
}
#endif

#endif /* BIFATTN_H */
