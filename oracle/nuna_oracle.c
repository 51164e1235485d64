/*
 * nuna_oracle.c -- plain CPU oracle for the collective copy/reduce semantics.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path links, loads or calls
 * this file; only the test suite, the smoke check and the benchmark's CPU
 * baseline leg do.  It shares no code, header, table or helper with the HIP
 * library: it is written from the definitions of the collectives (Sec. 2.1 of
 * the paper: all-gather, all-reduce, all-to-all as the common AI patterns;
 * reduce-scatter + all-gather in tensor-parallel traces, same section) and the
 * accumulation rule fixed for this path (fp32 accumulation of bf16 inputs,
 * ranks summed in ascending order, one rounding at the end).
 *
 * Every routine is a direct, slow, element-at-a-time loop.  No blocking, no
 * vectorisation tricks, no reordering of the sum.  Built with
 * -O1 -ffp-contract=off -fno-fast-math so that every float addition below is
 * exactly one IEEE-754 binary32 round-to-nearest-even addition.
 *
 * Data types: code 0 = fp32 (4-byte IEEE binary32), code 1 = bf16 (2-byte
 * bfloat16 bit patterns: the upper half of a binary32).
 *
 * Pins (what ties these routines to something other than themselves) live in
 * tests/test_oracle_pins.py: numpy's sequential add.accumulate, torch's
 * fp32->bf16 conversion over all 2^32 patterns, a from-the-definition fp64
 * round-to-nearest-even, exact integer sums, one-hot and constant closed
 * forms, the recursive-summation error bound against exact (fsum) sums,
 * all-gather(reduce-scatter) == all-reduce, and a brute-force Python
 * enumeration of the all-to-all routing on tiny inputs.
 */
#include <stdint.h>
#include <stddef.h>
#include <string.h>
#include <stdlib.h>

#define ORC_F32 0
#define ORC_BF16 1

/* ---- bf16 <-> fp32 ------------------------------------------------------ */

/* Widening bf16 -> fp32 is exact: the 16 bf16 bits become the upper half. */
static float orc_bf16_to_f32(uint16_t h)
{
    uint32_t u = ((uint32_t)h) << 16;
    float f;
    memcpy(&f, &u, sizeof f);
    return f;
}

/* Narrowing fp32 -> bf16 with round-to-nearest, ties-to-even on the 16
 * dropped mantissa bits.  A NaN stays a NaN: its sign and upper payload bits
 * are kept and the quiet bit is forced on.  Overflow past the largest finite
 * bf16 rounds to infinity, as round-to-nearest requires. */
static uint16_t orc_f32_to_bf16(float f)
{
    uint32_t u;
    memcpy(&u, &f, sizeof u);
    if ((u & 0x7fffffffu) > 0x7f800000u)
        return (uint16_t)((u >> 16) | 0x0040u);
    uint32_t upper = u >> 16;
    uint32_t lower = u & 0xffffu;
    /* lower > half: round up; lower < half: round down; tie: round to the even upper. */
    if (lower > 0x8000u || (lower == 0x8000u && (upper & 1u)))
        upper += 1u;
    return (uint16_t)upper;
}

uint16_t oracle_f32_to_bf16(float f) { return orc_f32_to_bf16(f); }
float oracle_bf16_to_f32(uint16_t h) { return orc_bf16_to_f32(h); }

/* Narrow a whole array (used by the exhaustive rounding pin). */
void oracle_f32_to_bf16_array(const float* x, uint16_t* y, size_t n)
{
    for (size_t i = 0; i < n; ++i) y[i] = orc_f32_to_bf16(x[i]);
}

static float orc_load(const void* buf, int dtype, size_t i)
{
    if (dtype == ORC_F32) return ((const float*)buf)[i];
    return orc_bf16_to_f32(((const uint16_t*)buf)[i]);
}

static void orc_store(void* buf, int dtype, size_t i, float v)
{
    if (dtype == ORC_F32) ((float*)buf)[i] = v;
    else ((uint16_t*)buf)[i] = orc_f32_to_bf16(v);
}

static size_t orc_esize(int dtype) { return dtype == ORC_F32 ? 4u : 2u; }

/* ---- all-reduce --------------------------------------------------------- */

/* The fp32 accumulator of element i: start from rank 0's value, then add
 * ranks 1, 2, ..., P-1 in that order, one fp32 rounding per addition. */
static float orc_sum_ascending(const void* const* in, int P, int dtype, size_t i)
{
    float acc = orc_load(in[0], dtype, i);
    for (int r = 1; r < P; ++r) acc = acc + orc_load(in[r], dtype, i);
    return acc;
}

/* All-reduce (sum): every destination buffer d receives, for every element
 * i, the ascending-rank fp32 sum narrowed once to the buffer's dtype.  The
 * result is the same whether the collective runs one-shot or as
 * reduce-scatter followed by all-gather.  In-place use (out[r] == in[r]) is
 * allowed: element i is fully read before it is written. */
int oracle_allreduce(int P, size_t n, int dtype, const void* const* in, void* const* out)
{
    if (P < 1 || (dtype != ORC_F32 && dtype != ORC_BF16)) return 1;
    for (size_t i = 0; i < n; ++i) {
        float acc = orc_sum_ascending(in, P, dtype, i);
        for (int d = 0; d < P; ++d) orc_store(out[d], dtype, i, acc);
    }
    return 0;
}

/* The fp32 accumulator itself, before narrowing (used for error-bound pins
 * and for the stated tolerance on other summation orders). */
int oracle_allreduce_acc_f32(int P, size_t n, int dtype, const void* const* in, float* acc_out)
{
    if (P < 1 || (dtype != ORC_F32 && dtype != ORC_BF16)) return 1;
    for (size_t i = 0; i < n; ++i) acc_out[i] = orc_sum_ascending(in, P, dtype, i);
    return 0;
}

/* ---- reduce-scatter ----------------------------------------------------- */

/* Each input buffer holds P*m elements; rank r owns the contiguous shard
 * [r*m, (r+1)*m).  out[r][j] = narrow(sum over q ascending of in[q][r*m+j]). */
int oracle_reduce_scatter(int P, size_t m, int dtype, const void* const* in, void* const* out)
{
    if (P < 1 || (dtype != ORC_F32 && dtype != ORC_BF16)) return 1;
    for (int r = 0; r < P; ++r) {
        for (size_t j = 0; j < m; ++j) {
            size_t i = (size_t)r * m + j;
            float acc = orc_sum_ascending(in, P, dtype, i);
            orc_store(out[r], dtype, j, acc);
        }
    }
    return 0;
}

/* ---- all-gather --------------------------------------------------------- */

/* Each input holds m elements; out[d][r*m + j] = in[r][j] for every d, as a
 * copy of the element's bytes (no float round trip). */
int oracle_all_gather(int P, size_t m, int dtype, const void* const* in, void* const* out)
{
    if (P < 1 || (dtype != ORC_F32 && dtype != ORC_BF16)) return 1;
    size_t es = orc_esize(dtype);
    for (int d = 0; d < P; ++d) {
        for (int r = 0; r < P; ++r) {
            const unsigned char* src = (const unsigned char*)in[r];
            unsigned char* dst = (unsigned char*)out[d] + (size_t)r * m * es;
            if (src == dst) continue; /* in-place shard: already there */
            for (size_t j = 0; j < m; ++j)
                for (size_t b = 0; b < es; ++b) dst[j * es + b] = src[j * es + b];
        }
    }
    return 0;
}

/* ---- all-to-all dispatch (MoE token routing) ---------------------------- */

/* Expert e lives on rank e / (E/P) (contiguous blocks of experts per rank).
 * Token t of source rank s is sent once to every distinct rank that owns one
 * of its top-k experts.  recv[d] lists, for s = 0..P-1 ascending and within
 * each s for t = 0..T-1 ascending, the rows (s, t) that go to d.
 *
 * oracle_a2a_counts fills rows[d] = number of rows rank d receives.
 * oracle_a2a_map fills, for one destination d, the (src rank, src token) of
 * each received row in receive order; it returns the number written. */
static int orc_token_goes_to(const int32_t* topk, int P, int T, int k, int E, int s, int t, int d)
{
    int per = E / P;
    const int32_t* ex = topk + ((size_t)s * T + t) * k;
    for (int j = 0; j < k; ++j)
        if (ex[j] / per == d) return 1;
    return 0;
}

int oracle_a2a_counts(int P, int T, int k, int E, const int32_t* topk, int64_t* rows)
{
    if (P < 1 || T < 0 || k < 1 || E < P || E % P != 0) return 1;
    for (int d = 0; d < P; ++d) {
        int64_t c = 0;
        for (int s = 0; s < P; ++s)
            for (int t = 0; t < T; ++t)
                c += orc_token_goes_to(topk, P, T, k, E, s, t, d);
        rows[d] = c;
    }
    return 0;
}

int64_t oracle_a2a_map(int P, int T, int k, int E, const int32_t* topk, int d,
                       int32_t* src_rank, int32_t* src_token)
{
    int64_t j = 0;
    for (int s = 0; s < P; ++s)
        for (int t = 0; t < T; ++t)
            if (orc_token_goes_to(topk, P, T, k, E, s, t, d)) {
                src_rank[j] = s;
                src_token[j] = t;
                ++j;
            }
    return j;
}

/* Row copy: recv[d][j, :] = send[s][t, :] for the j-th row (s, t) of d's map.
 * row_bytes is the size of one token row.  recv[d] must hold rows[d] rows. */
int oracle_all_to_all(int P, int T, int k, int E, const int32_t* topk, size_t row_bytes,
                      const void* const* send, void* const* recv)
{
    if (P < 1 || T < 0 || k < 1 || E < P || E % P != 0) return 1;
    for (int d = 0; d < P; ++d) {
        int64_t j = 0;
        for (int s = 0; s < P; ++s)
            for (int t = 0; t < T; ++t)
                if (orc_token_goes_to(topk, P, T, k, E, s, t, d)) {
                    const unsigned char* src = (const unsigned char*)send[s] + (size_t)t * row_bytes;
                    unsigned char* dst = (unsigned char*)recv[d] + (size_t)j * row_bytes;
                    for (size_t b = 0; b < row_bytes; ++b) dst[b] = src[b];
                    ++j;
                }
    }
    return 0;
}

/* ---- all-to-all combine (MoE result collection) ------------------------- */

/* The reverse of the dispatch above: rank d holds one result row y[d][j]
 * for the j-th row it received.  Token t of source rank s collects the
 * results of every rank it was sent to:
 *     out[s][t, :] = narrow(sum over d ascending, d a destination of (s, t),
 *                           of y[d][j(s, t, d), :])
 * with the same fp32 accumulation and single rounding as the all-reduce
 * (the first term starts the sum).  j(s, t, d) is the receive position the
 * dispatch gave token (s, t) at rank d.  Every token has at least one
 * destination (k >= 1), so every output row is written.
 *
 * Weighted form (the top-k weighted sum that gives a MoE layer its output):
 * when `weights` is not NULL it holds P*T*P floats, weights[(s*T + t)*P + d]
 * scaling the row rank d returns for token (s, t); each term is then the
 * fp32 product w * y (rounded once) before it joins the sum.  With one
 * expert per rank (E == P) these are the router's gate weights. */
int oracle_a2a_combine(int P, int T, int k, int E, const int32_t* topk, size_t row_elems, int dtype,
                       const float* weights, const void* const* y, void* const* out)
{
    if (P < 1 || T < 0 || k < 1 || E < P || E % P != 0 || (dtype != ORC_F32 && dtype != ORC_BF16)) return 1;
    int64_t* pos = (int64_t*)malloc(sizeof(int64_t) * (size_t)P * (size_t)(T > 0 ? T : 1) * (size_t)P);
    int64_t* next = (int64_t*)calloc((size_t)P, sizeof(int64_t));
    if (!pos || !next) { free(pos); free(next); return 2; }
    /* receive position of (s, t) at each destination, -1 when not sent there */
    for (int s = 0; s < P; ++s)
        for (int t = 0; t < T; ++t)
            for (int d = 0; d < P; ++d) {
                size_t idx = ((size_t)s * T + t) * P + d;
                pos[idx] = orc_token_goes_to(topk, P, T, k, E, s, t, d) ? next[d]++ : -1;
            }
    for (int s = 0; s < P; ++s)
        for (int t = 0; t < T; ++t)
            for (size_t h = 0; h < row_elems; ++h) {
                int have = 0;
                float acc = 0.0f;
                for (int d = 0; d < P; ++d) {
                    int64_t j = pos[((size_t)s * T + t) * P + d];
                    if (j < 0) continue;
                    float v = orc_load(y[d], dtype, (size_t)j * row_elems + h);
                    if (weights) v = weights[((size_t)s * T + t) * P + d] * v;
                    acc = have ? acc + v : v;
                    have = 1;
                }
                orc_store(out[s], dtype, (size_t)t * row_elems + h, acc);
            }
    free(pos);
    free(next);
    return 0;
}

