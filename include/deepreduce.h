/*
 * deepreduce.h -- C ABI of the MI355X (gfx950) DeepReduce sparse-tensor codec.
 *
 * The codec follows Kostopoulou et al., "DeepReduce: A Sparse-tensor
 * Communication Framework for Distributed Deep Learning" (arXiv 2102.03112):
 * a gradient is sparsified (top-r, or the support of an inherently sparse
 * gradient), its index set is compressed with a Bloom filter (Section 4) and
 * decoded with the no-error policy P0 (Section 4, "No-error approach") or a
 * policy that codes only r of the positives (P1 of Section 4 and Section
 * 10.5; the deterministic policies of Section 10.4), and its values are
 * compressed by sorting them and fitting a piecewise
 * least-squares polynomial (Section 5), with a bit-packed reorder map
 * (Section 5.1).
 *
 * Conventions for every call below:
 *  - Pointers are DEVICE pointers unless the parameter name ends in _h.
 *  - Calls are asynchronous on `stream` (a hipStream_t passed as void*;
 *    NULL is the default stream), except the host-only helpers marked so.
 *    Arguments are validated on the host before anything is launched; an
 *    invalid argument returns DR_EINVAL and launches nothing.
 *  - Counts produced by one call and consumed by the next stay in device
 *    memory (`uint64_t*` device scalars), so calls chain without host syncs.
 *    An input count `n` comes with `n_cap`, the host-side capacity of the
 *    items behind it (it sizes grids and scratch): a call processes the
 *    first min(*n, n_cap) items, and its `flags_out` word (device,
 *    nullable) receives DR_FLAG_CAPACITY when *n exceeds n_cap, else 0.
 *    Items past n_cap are then NOT processed (a filter built from a cut
 *    list yields false negatives for them), so a caller whose count can
 *    exceed its capacity must check that word.  An output capacity `cap`
 *    works the other way: entries beyond it are dropped and the full count
 *    is still reported, so the caller detects overflow by comparing the
 *    count with the capacity after synchronising.
 *  - Indices are 0-based u32 (the paper's [d] is 1-based, Section 2), so a
 *    gradient tensor holds fewer than 2^32 elements.
 *  - The caller owns all memory.  Scratch comes from `ws`, at least
 *    dr_workspace_bytes() bytes, device memory aligned to 256 bytes; its
 *    contents are undefined between calls and it must not be shared by calls
 *    that run concurrently.  The library keeps no state between calls.
 *  - Non-finite gradient values are outside the codec's contract: the
 *    results are then unspecified but every kernel still terminates, and the
 *    round trip reports them in its flags word (DR_FLAG_NONFINITE).
 *  - Hash family: MurmurHash3_x86_32 of the 4-byte little-endian index with
 *    seeds 0..k-1; bit position floor(h * m / 2^32); bit p of the filter is
 *    bit (p mod 32) of 32-bit word p / 32.
 */
#ifndef DEEPREDUCE_H
#define DEEPREDUCE_H

#include <stddef.h>
#include <stdint.h>

#if defined(__GNUC__) || defined(__clang__)
#define DR_EXPORT __attribute__((visibility("default")))
#else
#define DR_EXPORT
#endif

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    DR_OK = 0,
    DR_EINVAL = -1,    /* invalid argument; nothing was launched */
    DR_ECAPACITY = -2, /* a capacity given on the host is too small */
    DR_EDEVICE = -3,   /* a HIP runtime call failed; see dr_last_error() */
    DR_ENOTSUP = -4    /* a requested option is not implemented */
} dr_status;

/* r sentinel: select every element that is not +-0 (an inherently sparse
 * gradient, Section 3 and the NCF experiment of Section 6.3). */
#define DR_R_NONZERO UINT64_MAX

#define DR_MAX_DEGREE 7      /* highest polynomial degree per segment */
#define DR_MAX_SEGMENTS 4096 /* most segments per tensor */
#define DR_MAX_TENSORS 65536 /* most tensors in one round trip */
#define DR_MAX_SUM_PAYLOADS 64 /* most payloads summed by one dr_payload_decode_sum */

/* Index policies (Section 4; Sections 10.4 and 10.5): which of the filter's
 * positives P (ascending) get a value.  P0 codes all of them.  The others
 * code r = min(n_selected, |P|) of them: P1 a pseudo-random r-subset (see
 * dr_config.seed), LEFTMOST / MIDDLE / RIGHTMOST the first r, the r starting
 * at rank floor((|P| - r) / 2), or the last r.  A positive that is not coded
 * is received as 0. */
#define DR_POLICY_P0 0u
#define DR_POLICY_RANDOM 1u
#define DR_POLICY_LEFTMOST 2u
#define DR_POLICY_MIDDLE 3u
#define DR_POLICY_RIGHTMOST 4u

/* Segmentation of the sorted values into runs fitted separately (Section 5,
 * "Piece-wise approximation").  EQUAL: runs of equal count (as in
 * dr_curvefit_encode).  CHORD: the paper's split at the point farthest from
 * the chord joining a run's end points: the values with the sign bit clear
 * and the others start as two runs (when n_seg >= 2 and each has at least
 * degree+1 values); then, while there are fewer than n_seg runs, the run
 * whose farthest allowed point lies farthest from its chord (ties: the
 * leftmost run) is split after that point, a split being allowed only where
 * both parts keep at least degree+1 values; it stops early when no allowed
 * point lies off its chord.  The distance |C[a] + m (i - a) - C[i]| with m =
 * (C[z] - C[a]) / (z - a) (run [a, z], C the sorted values as doubles) is
 * evaluated in double with one rounding per operation; ties to the smaller
 * rank. */
#define DR_SEG_EQUAL 0u
#define DR_SEG_CHORD 1u

/* Value model per run (Section 5).  POLY: the least-squares polynomial of
 * degree `degree` (see dr_curvefit_encode).  DEXP: y = a e^(b t) + c e^(d t)
 * on the same abscissa t in [-1, 1], coefficient row (a, b, c, d) (so a
 * record's D_eff is 3 and runs hold at least 4 values; `degree` is not
 * used).  The fit: rates (1, -1) with the amplitudes that solve the linear
 * least-squares problem for them (a = mean, c = 0 if it is singular), then
 * 40 Levenberg-Marquardt steps solving (J^T J + lambda diag(J^T J)) delta =
 * J^T r in double, the trial rates clamped to [-40, 40], a trial kept only
 * if it lowers the residual sum of squares (lambda from 1e-3, /10 on a kept
 * step, x10 otherwise).  Decoding evaluates a e^(bt) + c e^(dt) in double
 * on the fp32 row and rounds to fp32.  A tensor with fewer than 4 values is
 * coded with the polynomial through them (the header names the model
 * used). */
#define DR_FIT_POLY 0u
#define DR_FIT_DEXP 1u

/* Where the sender takes the values of the positives it codes (Section 4,
 * policy P0).  SPARSE: from the sparsified gradient g~, whose entries are
 * g at the selected indices and 0 elsewhere, so a false positive carries
 * the value 0 (the base definition of P0).  DENSE: from the dense gradient
 * g, so a false positive carries its own gradient value (the variant the
 * paper allows when the sparsifier leaves g accessible, as GRACE does). */
#define DR_VALUES_DENSE 0u
#define DR_VALUES_SPARSE 1u

/* Filter layouts (the position map of the k hash functions; Section 2 asks
 * only for k independent hash functions into the m-bit array).  STANDARD
 * (record hash id 1): bit floor(h_j(i) m / 2^32) for every j.  PARTITIONED
 * (record hash id 2): the array is cut into k parts, part j covering bits
 * [floor(j m / k), floor((j+1) m / k)), and hash j sets bit floor(j m / k) +
 * floor(h_j(i) q_j / 2^32) of its part (q_j bits).  Same m, k, hash and
 * seeds; each part's fill is about 1 - e^{-kn/m}, so the false-positive rate
 * is Lemma 2's (1 - e^{-kn/m})^k as for the standard layout.  The receiver
 * takes the layout from each record.  The query of a partitioned filter
 * reads its first parts, those of the first probes, from on-chip memory. */
#define DR_FILTER_STANDARD 0u
#define DR_FILTER_PARTITIONED 1u

/* Bits of the per-tensor flags word (slot 3 of counts_out). */
#define DR_FLAG_NONFINITE 1u    /* the tensor held NaN or Inf */
#define DR_FLAG_DEC_MISMATCH 2u /* receiver: the record is invalid, or its |P| differs from the header */
#define DR_FLAG_COUNT 4u        /* sender: the selection does not hold exactly r elements */
#define DR_FLAG_CAPACITY 8u     /* a device-side capacity was exceeded; the output is incomplete */
#define DR_FLAG_STALLED 16u     /* an internal bounded wait gave up; the output is wrong (a bug) */

/* ---------------------------------------------------------------------- */
/* Host-only helpers                                                       */
/* ---------------------------------------------------------------------- */

/* Bloom filter size and hash count for n_items and a target false-positive
 * rate fpr in (0, 1), from Remark 2 of Section 10.2 (m = -n ln(fpr)/(ln 2)^2,
 * k = -ln(fpr)/ln 2), rounded as: k = max(1, round(-ln fpr / ln 2));
 * m = 32 * ceil(ceil(n * C) / 32) with C = -ln(fpr) / (ln 2 * ln 2), at least
 * 32.  Returns DR_EINVAL for fpr outside (0, 1) or m >= 2^32. */
DR_EXPORT dr_status dr_bloom_params(uint64_t n_items, double fpr, uint64_t *m_bits_h, uint32_t *k_h);

/* Bits per reorder-map entry for n values (Section 5.1): the smallest
 * b >= 1 with 2^b >= n. */
DR_EXPORT uint32_t dr_sigma_bits(uint64_t n);

/* Scratch bytes sufficient for any call of this library on a gradient of at
 * most d elements split into at most n_tensors tensors. */
DR_EXPORT size_t dr_workspace_bytes(uint64_t d, uint64_t n_tensors);

/* Message of the last failure on the calling host thread ("" if none). */
DR_EXPORT const char *dr_last_error(void);

/* Host-only, no GPU needed.  Replays, for configuration cfg_h, the index
 * ranges that the kernels derive from the host's plan (the Bloom insert's
 * item chunks and partial slices, for the round trip's selection bitmap and
 * for dr_bloom_encode's index list; the probe pass's per-block tile ranges
 * for several grid sizes; the value sort's tiles for value counts from 0 to
 * each tensor's size) with the same arithmetic the kernels run, and checks
 * every range against the buffer it addresses.  *violations_h receives the
 * number of ranges that would leave their buffer (0 for a sound plan); when
 * it is not 0, dr_last_error() describes the first.  EINVAL: an invalid
 * cfg_h or a null violations_h. */
typedef struct dr_config dr_config;
DR_EXPORT dr_status dr_check_ranges(const dr_config *cfg_h, uint64_t *violations_h);

/* ---------------------------------------------------------------------- */
/* Sparsification (Section 2 "Sparsification"; Section 10.2)               */
/* ---------------------------------------------------------------------- */

/* Top-r: the indices of the r entries of g[0..d) of largest magnitude, ties
 * broken by smaller index, written in ascending index order to idx_out
 * (capacity r); val_out (nullable, capacity r) receives g at those indices;
 * *n_out (device) receives r.  With r == DR_R_NONZERO, every entry that is
 * not +-0 is selected instead, idx_out and val_out need capacity d, and
 * *n_out receives their number.  EINVAL: d >= 2^32, r > d, null pointers,
 * workspace too small. */
DR_EXPORT dr_status dr_sparsify_topr(const float *g, uint64_t d, uint64_t r, uint32_t *idx_out, float *val_out,
                           uint64_t *n_out, void *ws, size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------------- */
/* Bloom-filter index compression (Sections 2 and 4)                       */
/* ---------------------------------------------------------------------- */

/* Insert the *n (device count) indices idx[0..*n) into an m_bits-bit filter
 * with k hash functions: set bit h_j(x) for every x and j < k.  bits_out
 * receives all m_bits/32 words (the callee clears them first).  n_cap is
 * the capacity of idx: at most n_cap indices are inserted, and flags_out
 * (device, nullable) receives DR_FLAG_CAPACITY if *n > n_cap (see the
 * conventions above), else 0.  m_bits must be a positive multiple of 32
 * below 2^32; 1 <= k <= 32.  Indices must be below 2^32. */
DR_EXPORT dr_status dr_bloom_encode(const uint32_t *idx, const uint64_t *n, uint64_t n_cap, uint64_t m_bits, uint32_t k,
                          uint32_t *bits_out, uint64_t *flags_out, void *ws, size_t ws_bytes, void *stream);

/* Full-range query of policy P0 (Section 4): every i in [0, d) whose k bits
 * are all set in `bits`, written in ascending order to idx_out (at most cap
 * entries; the full count goes to *n_out, device).  True and false
 * positives are both reported; a filter never yields a false negative. */
DR_EXPORT dr_status dr_bloom_decode(const uint32_t *bits, uint64_t m_bits, uint32_t k, uint64_t d, uint32_t *idx_out,
                          uint64_t cap, uint64_t *n_out, void *ws, size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------------- */
/* Curve-fitting value compression (Section 5; reorder map Section 5.1)    */
/* ---------------------------------------------------------------------- */

/* Compress vals[0..*n) (device count; n_cap, the capacity of vals, bounds
 * it and flags_out, device and nullable, receives DR_FLAG_CAPACITY if *n >
 * n_cap, else 0, as the conventions above say): sort the values
 * in descending order (signed; +0 before -0; equal values keep their
 * order), split the sorted sequence into S_eff = min(n_seg, max(1,
 * floor(n/(degree+1)))) runs of equal count (run s holds sorted ranks
 * [floor(s n / S_eff), floor((s+1) n / S_eff))), and fit each run by least
 * squares with a polynomial of degree D_eff = degree (or n-1 if n < degree+1)
 * in t = (2j - (n_s - 1)) / (n_s - 1) for local rank j of n_s points (t = 0
 * when n_s = 1), solved in double precision.
 * coef_out (n_seg*(degree+1) floats) receives run s's coefficient of t^p at
 * [s*(degree+1) + p] rounded to fp32, zeros elsewhere.
 * sigma_out receives the reorder map sigma[q] = sorted rank of vals[q] in
 * b = dr_sigma_bits(n) bits per entry, entry q at bits [q b, (q+1) b) of the
 * LSB-first 32-bit word stream; capacity ceil(n_cap * dr_sigma_bits(n_cap)
 * / 32) words.  EINVAL: degree > DR_MAX_DEGREE, n_seg == 0 or
 * > DR_MAX_SEGMENTS, n_cap >= 2^32. */
DR_EXPORT dr_status dr_curvefit_encode(const float *vals, const uint64_t *n, uint64_t n_cap, uint32_t degree, uint32_t n_seg,
                             float *coef_out, uint32_t *sigma_out, uint64_t *flags_out, void *ws, size_t ws_bytes,
                             void *stream);

/* Reconstruct *n values from coef and sigma as written by
 * dr_curvefit_encode: value q is run s's polynomial, evaluated by Horner's
 * rule in double at the abscissa of rank sigma[q], rounded to fp32.  n_cap
 * is the capacity of vals_out: at most n_cap values are written, and
 * flags_out (device, nullable) receives DR_FLAG_CAPACITY if *n > n_cap,
 * else 0. */
DR_EXPORT dr_status dr_curvefit_decode(const float *coef, const uint32_t *sigma, const uint64_t *n, uint64_t n_cap,
                             uint32_t degree, uint32_t n_seg, float *vals_out, uint64_t *flags_out, void *ws,
                             size_t ws_bytes, void *stream);

/* ---------------------------------------------------------------------- */
/* The whole codec over a gradient split into tensors (Figure 3)           */
/* ---------------------------------------------------------------------- */

struct dr_config {
    uint64_t n_tensors;        /* >= 1, at most DR_MAX_TENSORS */
    const uint64_t *offsets_h; /* host, n_tensors+1 nondecreasing offsets, [0] = 0; tensor t is
                                  g[offsets_h[t] .. offsets_h[t+1]), fewer than 2^32 elements */
    uint64_t ratio_num;        /* top-r: r_t = ceil(d_t * ratio_num / ratio_den) <= d_t;         */
    uint64_t ratio_den;        /*   ratio_num == DR_R_NONZERO selects every nonzero instead      */
    double fpr;                /* Bloom target false-positive rate, in (0, 1)                    */
    uint32_t degree;           /* polynomial degree per run, <= DR_MAX_DEGREE                    */
    uint32_t n_seg;            /* runs per tensor, 1 .. DR_MAX_SEGMENTS; 0: from the sorted values,
                                  p + 1 runs with p = ceil(2 sqrt(M)) for degree >= 1 (Section 5,
                                  after Lemma 1) or ceil(M / sqrt(2) - 1) for degree 0 (Remark 4),
                                  M = |(C[0] - C[1]) - (C[n-2] - C[n-1])| in double, each ceiling
                                  taken as the smallest p >= 0 with p^2 >= 4M, resp.
                                  2 (p+1)^2 >= M^2; at most DR_MAX_SEGMENTS runs              */
    uint32_t policy;           /* DR_POLICY_*; the receiver takes it from each record's header   */
    uint32_t seed;             /* key of DR_POLICY_RANDOM (ignored by the others): positive q of
                                  P is coded iff pi(q) < r, as value number pi(q), where pi is a
                                  permutation of [0, |P|): a 4-round Feistel network on 2h-bit
                                  words (h = max(1, ceil(ceil(log2 |P|) / 2))) whose round j
                                  XORs MurmurHash3_x86_32(LE half, seed + j) mod 2^h into the
                                  other half, restricted to [0, |P|) by cycle walking */
    uint32_t segmentation;     /* DR_SEG_EQUAL or DR_SEG_CHORD                                   */
    uint32_t fit_model;        /* DR_FIT_POLY or DR_FIT_DEXP                                     */
    uint32_t value_source;     /* DR_VALUES_DENSE or DR_VALUES_SPARSE                            */
    uint32_t filter_layout;    /* DR_FILTER_STANDARD or DR_FILTER_PARTITIONED                    */
};

/* Payload container (Figure 3's "container"): one record per tensor at byte
 * offset rec_off_h[t] (multiples of 256) of the payload buffer.  A record is
 * a 64-byte header followed by the filter words, the fp32 coefficients of
 * the S_eff x (D_eff+1) fitted polynomials, under DR_SEG_CHORD the S_eff - 1
 * u32 starts of runs 1 .. S_eff-1 (sorted ranks, ascending), and the packed
 * reorder map, each section padded to 4 bytes and packed back to back.
 * Header layout: 16 little-endian u32 words: magic 0x31435244 ("DRC1"),
 * header bytes (64), d, n_selected, n_positives (|P|), n_values (values
 * coded: |P| under P0), m_bits, k, hash id (MurmurHash3_x86_32 with seeds
 * 0..k-1; 1 = standard filter layout, 2 = partitioned), policy,
 * seed, D_eff, S_eff, sigma bits, record bytes (header + sections; what
 * would be sent), segmentation (DR_SEG_*) | value model (DR_FIT_*) << 8 |
 * value source (DR_VALUES_*) << 16.
 * Returns the total payload capacity in bytes; fills rec_off_h (nullable,
 * n_tensors+1 entries) with the record offsets and the end.  Returns 0 for
 * an invalid configuration. */
DR_EXPORT size_t dr_payload_layout(const dr_config *cfg_h, uint64_t *rec_off_h);

/* Sender side over the whole gradient g: per tensor, select (top-r or
 * support), insert into a Bloom filter sized by dr_bloom_params, run the
 * full-range query (P), let the policy pick the positives to code, take
 * their values from the dense gradient (V = g[P] under P0) or from the
 * sparsified one (V = g~[P]: 0 at false positives), as cfg_h->value_source
 * says (Section 4), sort and fit V, and write the record into `payload`
 * (capacity
 * payload_bytes, at least dr_payload_layout()).  counts_out (device,
 * nullable) receives 4 u64 per tensor: n_selected, |P|, 0, flags. */
DR_EXPORT dr_status dr_payload_encode(const float *g, const dr_config *cfg_h, uint8_t *payload, size_t payload_bytes,
                            uint64_t *counts_out, void *ws, size_t ws_bytes, void *stream);

/* Receiver side: from the payload alone, recover P by the full-range query
 * of each tensor's filter, evaluate the fitted values at the ranks the
 * reorder map gives (through the record's policy: a positive the policy
 * did not code is 0), and write the dense gradient dense_out (d floats,
 * zero off P).  idx_out / val_out (nullable, d entries) receive tensor t's
 * positives (local indices) and their values at [offsets_h[t], offsets_h[t]
 * + |P_t|).  counts_out (nullable): slot 2 of each tensor receives the
 * receiver's |P|; slot 3 gains DR_FLAG_DEC_MISMATCH if it disagrees with
 * the header or the record is invalid (an invalid record decodes as empty). */
DR_EXPORT dr_status dr_payload_decode(const uint8_t *payload, const dr_config *cfg_h, float *dense_out, uint32_t *idx_out,
                            float *val_out, uint64_t *counts_out, void *ws, size_t ws_bytes, void *stream);

/* Receiver side of a data-parallel step (Section 2, "Compressed distributed
 * training via SGD": the workers' compressed gradients are averaged; Section
 * 6.4 exchanges DeepReduce payloads by all-gather, so each worker decodes
 * all of them).  payloads_h (host array of n_payloads device pointers, 1 ..
 * DR_MAX_SUM_PAYLOADS) holds payloads written by dr_payload_encode with the
 * tensor layout of cfg_h (their records at dr_payload_layout's offsets).
 * dense_out (d floats) receives scale * (g_0 + g_1 + ... + g_{n-1}), where
 * g_p is the dense gradient dr_payload_decode rebuilds from payload p: the
 * terms of each element are added in fp32 in payload order, starting from
 * +0, and the sum is then multiplied by scale in fp32 (scale = 1/n gives the
 * average).  One pass over the dense gradient writes it once.  counts_out
 * (device, nullable) receives 4 u64 per payload and tensor, payload-major:
 * 0, 0, the receiver's |P|, flags (DR_FLAG_DEC_MISMATCH as for
 * dr_payload_decode).  The workspace needs dr_workspace_bytes(d,
 * n_tensors) bytes.  EINVAL: n_payloads out of range, a null payload
 * pointer, dense_out null with d > 0, scale not finite, an invalid cfg_h,
 * workspace too small. */
DR_EXPORT dr_status dr_payload_decode_sum(const uint8_t *const *payloads_h, uint32_t n_payloads, const dr_config *cfg_h,
                                          float scale, float *dense_out, uint64_t *counts_out, void *ws,
                                          size_t ws_bytes, void *stream);

/* dr_payload_encode followed by dr_payload_decode: one codec round trip of
 * the whole gradient, with the same results.  The receiver's query pass
 * needs only the records' headers and filters, so once the sender's query
 * pass has written them the library runs it on a second stream of its own
 * (one per device, created on first use) while the sender emits, sorts and
 * fits its values (the receiver's set-up runs there from the start);
 * the second stream waits for `stream` and `stream` waits for it before the
 * receiver's last pass, so the call stays ordered on `stream` (also under
 * graph capture).  This needs room in `ws` for the receiver's own state
 * after the sender's (dr_workspace_bytes leaves it for the usual layouts);
 * otherwise, and with chord segmentation or the heuristic run count, the
 * two sides run one after the other. */
DR_EXPORT dr_status dr_roundtrip(const float *g, const dr_config *cfg_h, uint8_t *payload, size_t payload_bytes,
                       float *dense_out, uint32_t *idx_out, float *val_out, uint64_t *counts_out, void *ws,
                       size_t ws_bytes, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid hipMalloc): the same
 * round trip as dr_roundtrip, with the same results, but its scratch is a
 * static device array of the library, DR_STATIC_SCRATCH_BYTES bytes on each
 * GPU it runs on (allocated when the library's code is loaded there and held
 * until the process ends), instead of a caller's workspace.  The caller
 * still passes the gradient, the payload and the outputs.  The sender and
 * the receiver run one after the other on `stream`; the call launches only
 * kernels (no second stream, no event, no hipMalloc, hipFree or memset; keep
 * per-kernel tracing off).  DR_ECAPACITY, before anything is launched, if
 * the configuration needs more scratch than the array holds: 64 MiB covers
 * the round trip of gradients up to about one million elements.  Every call
 * on one GPU shares that GPU's array, which keeps the last call's contents
 * (each call clears what it needs cleared): calls that overlap on one GPU
 * (other host threads, or other streams not ordered with this one) race. */
#define DR_STATIC_SCRATCH_BYTES (64ull << 20)
DR_EXPORT dr_status dr_roundtrip_static(const float *g, const dr_config *cfg_h, uint8_t *payload,
                                        size_t payload_bytes, float *dense_out, uint32_t *idx_out, float *val_out,
                                        uint64_t *counts_out, void *stream);

/* ---------------------------------------------------------------------- */
/* Per-kernel timing (the paper reports encode/decode wall time, Section   */
/* 6.4; this breaks it down by kernel)                                     */
/* ---------------------------------------------------------------------- */

/* Start timing on the calling host thread: an event is recorded on `stream`
 * now, at the start of every later entry point, and after every kernel the
 * library launches from this thread, until dr_trace_end.  Events add a few
 * microseconds per kernel; time the codec itself with tracing off.
 * EINVAL if tracing is already on for this thread. */
DR_EXPORT dr_status dr_trace_begin(void *stream);

/* Stop timing, wait for the recorded events, and write one line per kernel
 * name into buf_h (NUL-terminated, truncated to buf_bytes): "<kernel>
 * <launches> <total milliseconds>\n".  A kernel's time runs from the
 * previous event on its own stream; dr_roundtrip runs part of the receiver
 * on a second stream beside the sender, so the times of kernels on the two
 * streams overlap and may add up to more than the elapsed time.  Idle time
 * between entry points is not attributed to any kernel.  EINVAL if tracing
 * was not begun. */
DR_EXPORT dr_status dr_trace_end(char *buf_h, size_t buf_bytes);

#ifdef __cplusplus
}
#endif

#endif /* DEEPREDUCE_H */
