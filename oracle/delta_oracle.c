/*
 * Plain CPU oracle for the lossless sparse delta checkpoint of AuroraRL
 * (arXiv 2602.11456).
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or
 * call this file: only the test suite, the smoke check and the CPU baseline
 * leg of the benchmark use it.  It shares no code, header, table or helper
 * with the GPU library; it includes nothing but the C standard library.
 *
 * Every function is the plain definition written out as one sequential loop
 * over elements, with no blocking, vectorisation or reordering:
 *
 *   extract        Sec. 5.1 "Sparse encoding": each tensor's delta is
 *                  flattened to a 1-D index space and its non-zeros are kept
 *                  as two 1-D arrays, idx and val, with a fixed-width int32 or
 *                  int64 index and a bfloat16 value.  The index array is
 *                  sorted (the gap encoding of Sec. 5.1 is defined on it).
 *                  A position is kept when its bf16 bit pattern changed; the
 *                  value kept is the updated bf16 word (reading: a bitwise
 *                  compare and an assignment scatter are what make the
 *                  round trip lossless, Sec. 5.1 "Lossless precision").
 *   extract_multi  Sec. 5.1: several tensors share one linear index space by
 *                  adding a fixed block offset (the sum of the sizes of the
 *                  tensors before it) to each tensor's own linear indices.
 *   apply          Sec. 5.1 / Sec. 5.2: the actor writes the streams into the
 *                  parameter's flat storage in place.
 *   gap + LEB128   Sec. 5.1 and Fig. "Delta checkpoint index encoding": the
 *                  sorted index array keeps its first entry as-is and every
 *                  later entry as the difference from its predecessor; each
 *                  number is then written as unsigned LEB128 (7 payload bits
 *                  per byte, least significant group first, high bit set on
 *                  every byte but the last).
 *   xxh64          Sec. 5.1 / Sec. 5.2: every delta checkpoint carries an
 *                  integrity hash and is cut into segments verified against
 *                  it.  The hash is XXH64 (Y. Collet, "xxHash fast digest
 *                  algorithm", specification v0.1.1), written out from that
 *                  specification: four 64-bit accumulators over 32-byte
 *                  stripes, a merge, the tail in 8/4/1-byte steps, and the
 *                  final avalanche.
 *   compose        Sec. 5.4 "Version-predicate join and delta catch-up": a
 *                  worker K versions behind replays the missed deltas in
 *                  order.  Apply assigns, so that replay equals one delta
 *                  holding every index of the chain with the value of the
 *                  newest delta that has it (merge of the sorted streams,
 *                  the last writer wins).
 *
 * Conventions shared with the library's C ABI (they are the ABI's contract,
 * restated here, not code shared with it): bf16 words travel as raw uint16
 * bit patterns; "count" results are always the true number of entries even
 * when it exceeds the caller's capacity, and only the first `capacity`
 * entries are written.
 */
#include <pthread.h>
#include <stdint.h>
#include <stddef.h>
#include <stdlib.h>

/* ------------------------------------------------------------------ */
/* extract: one tensor, local indices                                  */
/* ------------------------------------------------------------------ */

/* Sec. 5.1 "Sparse encoding", int64 index variant. */
uint64_t oracle_extract_i64(const uint16_t *prev, const uint16_t *next,
                            uint64_t n, int64_t *idx, uint16_t *val,
                            uint64_t capacity)
{
    uint64_t count = 0;
    for (uint64_t i = 0; i < n; ++i) {
        if (prev[i] != next[i]) {
            if (count < capacity) {
                idx[count] = (int64_t)i;
                val[count] = next[i];
            }
            ++count;
        }
    }
    return count;
}

/* Sec. 5.1 "Sparse encoding", int32 index variant (caller guarantees that
 * n - 1 fits in int32). */
uint64_t oracle_extract_i32(const uint16_t *prev, const uint16_t *next,
                            uint64_t n, int32_t *idx, uint16_t *val,
                            uint64_t capacity)
{
    uint64_t count = 0;
    for (uint64_t i = 0; i < n; ++i) {
        if (prev[i] != next[i]) {
            if (count < capacity) {
                idx[count] = (int32_t)i;
                val[count] = next[i];
            }
            ++count;
        }
    }
    return count;
}

/* ------------------------------------------------------------------ */
/* extract_multi: a list of tensors in one global index space          */
/* ------------------------------------------------------------------ */

/* Sec. 5.1: tensor t contributes global index base_t + i, where base_t is
 * the total size of tensors 0..t-1.  tensor_offsets (T+1 entries, may be
 * NULL) receives the output position of each tensor's first entry, and the
 * total at index T. */
uint64_t oracle_extract_multi(const uint16_t *const *prevs,
                              const uint16_t *const *nexts,
                              const uint64_t *numels, int32_t num_tensors,
                              int64_t *idx, uint16_t *val, uint64_t capacity,
                              uint64_t *tensor_offsets)
{
    uint64_t count = 0;
    uint64_t base = 0;
    for (int32_t t = 0; t < num_tensors; ++t) {
        if (tensor_offsets)
            tensor_offsets[t] = count;
        const uint16_t *p = prevs[t];
        const uint16_t *q = nexts[t];
        for (uint64_t i = 0; i < numels[t]; ++i) {
            if (p[i] != q[i]) {
                if (count < capacity) {
                    idx[count] = (int64_t)(base + i);
                    val[count] = q[i];
                }
                ++count;
            }
        }
        base += numels[t];
    }
    if (tensor_offsets)
        tensor_offsets[num_tensors] = count;
    return count;
}

/* ------------------------------------------------------------------ */
/* extract_multi on several host threads (CPU baseline timing only)     */
/* ------------------------------------------------------------------ */

/* One thread's share: the global index range [lo, hi) scanned with the
 * plain loop of oracle_extract_multi into a list of its own, and the
 * number of its entries in each tensor. */
struct oracle_range_job {
    const uint16_t *const *prevs;
    const uint16_t *const *nexts;
    const uint64_t *numels;
    int32_t num_tensors;
    uint64_t lo, hi;
    int64_t *idx;
    uint16_t *val;
    uint64_t count, room;
    uint64_t *tensor_counts;
    int failed;
};

static void *oracle_range_scan(void *arg)
{
    struct oracle_range_job *j = (struct oracle_range_job *)arg;
    uint64_t base = 0;
    for (int32_t t = 0; t < j->num_tensors; ++t) {
        const uint64_t n = j->numels[t];
        if (j->hi > base && j->lo < base + n) {
            const uint64_t a = j->lo > base ? j->lo - base : 0;
            const uint64_t b = j->hi < base + n ? j->hi - base : n;
            const uint16_t *p = j->prevs[t];
            const uint16_t *q = j->nexts[t];
            for (uint64_t i = a; i < b; ++i) {
                if (p[i] != q[i]) {
                    if (j->count == j->room) {
                        const uint64_t room = j->room ? 2 * j->room : 4096;
                        int64_t *ni = (int64_t *)realloc(j->idx, room * sizeof(int64_t));
                        if (ni) j->idx = ni;
                        uint16_t *nv = (uint16_t *)realloc(j->val, room * sizeof(uint16_t));
                        if (nv) j->val = nv;
                        if (!ni || !nv) {
                            j->failed = 1;
                            return NULL;
                        }
                        j->room = room;
                    }
                    j->idx[j->count] = (int64_t)(base + i);
                    j->val[j->count] = q[i];
                    ++j->count;
                    ++j->tensor_counts[t];
                }
            }
        }
        base += n;
    }
    return NULL;
}

/* The result of oracle_extract_multi, computed by `num_threads` POSIX
 * threads for timing the CPU on all its cores: the global index space is
 * cut into num_threads contiguous ranges of equal size, every thread runs
 * the plain loop over its range into its own list, and the lists are
 * concatenated in range order (the ranges are disjoint and ascending, so
 * this is the definition's sorted list).  At most 256 threads are used.
 * Returns UINT64_MAX if a thread or its memory could not be had. */
uint64_t oracle_extract_multi_threaded(const uint16_t *const *prevs,
                                       const uint16_t *const *nexts,
                                       const uint64_t *numels, int32_t num_tensors,
                                       int64_t *idx, uint16_t *val, uint64_t capacity,
                                       uint64_t *tensor_offsets, int32_t num_threads)
{
    if (num_threads < 1)
        num_threads = 1;
    if (num_threads > 256)
        num_threads = 256;
    uint64_t total = 0;
    for (int32_t t = 0; t < num_tensors; ++t)
        total += numels[t];
    const size_t T = num_tensors > 0 ? (size_t)num_tensors : 1;
    struct oracle_range_job *jobs =
        (struct oracle_range_job *)calloc((size_t)num_threads, sizeof(*jobs));
    pthread_t *tids = (pthread_t *)calloc((size_t)num_threads, sizeof(pthread_t));
    char *started = (char *)calloc((size_t)num_threads, 1);
    uint64_t *tcounts = (uint64_t *)calloc((size_t)num_threads * T, sizeof(uint64_t));
    uint64_t result = UINT64_MAX;
    if (!jobs || !tids || !started || !tcounts)
        goto done;
    for (int32_t r = 0; r < num_threads; ++r) {
        struct oracle_range_job *j = &jobs[r];
        j->prevs = prevs;
        j->nexts = nexts;
        j->numels = numels;
        j->num_tensors = num_tensors;
        j->lo = (uint64_t)((unsigned __int128)total * (uint64_t)r / (uint64_t)num_threads);
        j->hi = (uint64_t)((unsigned __int128)total * (uint64_t)(r + 1) / (uint64_t)num_threads);
        j->tensor_counts = tcounts + (size_t)r * T;
        if (pthread_create(&tids[r], NULL, oracle_range_scan, j) != 0)
            goto join;
        started[r] = 1;
    }
join:
    for (int32_t r = 0; r < num_threads; ++r)
        if (started[r])
            pthread_join(tids[r], NULL);
    for (int32_t r = 0; r < num_threads; ++r)
        if (!started[r] || jobs[r].failed)
            goto done;
    /* concatenate in range order */
    uint64_t count = 0;
    for (int32_t r = 0; r < num_threads; ++r) {
        for (uint64_t k = 0; k < jobs[r].count; ++k) {
            if (count < capacity) {
                idx[count] = jobs[r].idx[k];
                val[count] = jobs[r].val[k];
            }
            ++count;
        }
    }
    if (tensor_offsets) {
        uint64_t before = 0;
        for (int32_t t = 0; t < num_tensors; ++t) {
            tensor_offsets[t] = before;
            for (int32_t r = 0; r < num_threads; ++r)
                before += tcounts[(size_t)r * T + (size_t)t];
        }
        tensor_offsets[num_tensors] = before;
    }
    result = count;
done:
    if (jobs)
        for (int32_t r = 0; r < num_threads; ++r) {
            free(jobs[r].idx);
            free(jobs[r].val);
        }
    free(jobs);
    free(tids);
    free(started);
    free(tcounts);
    return result;
}

/* ------------------------------------------------------------------ */
/* apply: in-place scatter of the value stream                          */
/* ------------------------------------------------------------------ */

/* Sec. 5.1 / 5.2: w[idx[k]] = val[k].  Entries whose index is outside
 * [0, n) are skipped; the return value is how many were skipped. */
uint64_t oracle_apply_i64(uint16_t *w, uint64_t n, const int64_t *idx,
                          const uint16_t *val, uint64_t count)
{
    uint64_t bad = 0;
    for (uint64_t k = 0; k < count; ++k) {
        if (idx[k] < 0 || (uint64_t)idx[k] >= n) {
            ++bad;
            continue;
        }
        w[idx[k]] = val[k];
    }
    return bad;
}

uint64_t oracle_apply_i32(uint16_t *w, uint64_t n, const int32_t *idx,
                          const uint16_t *val, uint64_t count)
{
    uint64_t bad = 0;
    for (uint64_t k = 0; k < count; ++k) {
        if (idx[k] < 0 || (uint64_t)idx[k] >= n) {
            ++bad;
            continue;
        }
        w[idx[k]] = val[k];
    }
    return bad;
}

/* Sec. 5.1: a global index g belongs to the tensor t with
 * base_t <= g < base_t + n_t, at local position g - base_t.  The tensor is
 * found by scanning the bases in order, so any index order is accepted. */
uint64_t oracle_apply_multi(uint16_t *const *ws, const uint64_t *numels,
                            int32_t num_tensors, const int64_t *idx,
                            const uint16_t *val, uint64_t count)
{
    uint64_t bad = 0;
    for (uint64_t k = 0; k < count; ++k) {
        int64_t g = idx[k];
        int found = 0;
        if (g >= 0) {
            uint64_t base = 0;
            for (int32_t t = 0; t < num_tensors; ++t) {
                if ((uint64_t)g < base + numels[t]) {
                    ws[t][(uint64_t)g - base] = val[k];
                    found = 1;
                    break;
                }
                base += numels[t];
            }
        }
        if (!found)
            ++bad;
    }
    return bad;
}

/* ------------------------------------------------------------------ */
/* gap + unsigned LEB128 index encoding                                */
/* ------------------------------------------------------------------ */

/* Sec. 5.1: gaps of a sorted index array, first entry kept as-is.
 * Returns 0 on success, 1 if the input is not strictly increasing or has a
 * negative first entry. */
int oracle_gaps(const int64_t *idx, uint64_t count, uint64_t *gaps)
{
    for (uint64_t k = 0; k < count; ++k) {
        if (k == 0) {
            if (idx[0] < 0)
                return 1;
            gaps[0] = (uint64_t)idx[0];
        } else {
            if (idx[k] <= idx[k - 1])
                return 1;
            gaps[k] = (uint64_t)(idx[k] - idx[k - 1]);
        }
    }
    return 0;
}

/* Unsigned LEB128 of one number: 7-bit groups, least significant first,
 * continuation flag (0x80) on every byte except the last.  Writes at most
 * 10 bytes; returns the number of bytes. */
static int leb128_put(uint64_t v, uint8_t *out)
{
    int nb = 0;
    do {
        uint8_t byte = (uint8_t)(v & 0x7F);
        v >>= 7;
        if (v != 0)
            byte |= 0x80;
        out[nb++] = byte;
    } while (v != 0);
    return nb;
}

/* Encodes the gaps of idx as one LEB128 byte stream.  Returns the true
 * byte length (only the first `capacity` bytes are written), or
 * UINT64_MAX if idx is not strictly increasing / non-negative. */
uint64_t oracle_leb128_encode(const int64_t *idx, uint64_t count,
                              uint8_t *out, uint64_t capacity)
{
    uint64_t len = 0;
    int64_t prev = 0;
    for (uint64_t k = 0; k < count; ++k) {
        uint64_t gap;
        if (k == 0) {
            if (idx[0] < 0)
                return UINT64_MAX;
            gap = (uint64_t)idx[0];
        } else {
            if (idx[k] <= prev)
                return UINT64_MAX;
            gap = (uint64_t)(idx[k] - prev);
        }
        prev = idx[k];
        uint8_t tmp[10];
        int nb = leb128_put(gap, tmp);
        for (int b = 0; b < nb; ++b) {
            if (len < capacity)
                out[len] = tmp[b];
            ++len;
        }
    }
    return len;
}

/* Decodes a LEB128 gap stream back to absolute indices (running sum of the
 * gaps).  Returns the number of indices decoded (only the first
 * `capacity` written), or UINT64_MAX if the stream ends inside a number or
 * a number needs more than 64 bits. */
uint64_t oracle_leb128_decode(const uint8_t *in, uint64_t nbytes,
                              int64_t *idx, uint64_t capacity)
{
    uint64_t count = 0;
    uint64_t pos = 0;
    uint64_t acc = 0;
    while (pos < nbytes) {
        uint64_t v = 0;
        int shift = 0;
        for (;;) {
            if (pos >= nbytes)
                return UINT64_MAX;
            uint8_t byte = in[pos++];
            uint64_t payload = (uint64_t)(byte & 0x7F);
            if (shift > 63 || (shift == 63 && payload > 1))
                return UINT64_MAX;
            v |= payload << shift;
            shift += 7;
            if ((byte & 0x80) == 0)
                break;
        }
        acc = (count == 0) ? v : acc + v;
        if (count < capacity)
            idx[count] = (int64_t)acc;
        ++count;
    }
    return count;
}

/* ------------------------------------------------------------------ */
/* delta chain composition                                             */
/* ------------------------------------------------------------------ */

/* Sec. 5.4: the deltas D_1 .. D_K (oldest first, each with a strictly
 * increasing index stream) as one delta.  K-pointer merge: take the
 * smallest index that any stream has not passed yet, keep the value of the
 * newest stream that holds it, and step past it in every stream that holds
 * it.  Returns the true count (only the first `capacity` entries written),
 * or UINT64_MAX if some stream is not strictly increasing. */
uint64_t oracle_compose(const int64_t *const *idxs, const uint16_t *const *vals,
                        const uint64_t *counts, int32_t num_deltas, int64_t *out_idx,
                        uint16_t *out_val, uint64_t capacity)
{
    for (int32_t d = 0; d < num_deltas; ++d)
        for (uint64_t k = 1; k < counts[d]; ++k)
            if (idxs[d][k] <= idxs[d][k - 1])
                return UINT64_MAX;
    uint64_t *pos = calloc(num_deltas > 0 ? (size_t)num_deltas : 1, sizeof(uint64_t));
    if (!pos)
        return UINT64_MAX;
    uint64_t count = 0;
    for (;;) {
        int found = 0;
        int64_t smallest = 0;
        for (int32_t d = 0; d < num_deltas; ++d) {
            if (pos[d] < counts[d] && (!found || idxs[d][pos[d]] < smallest)) {
                smallest = idxs[d][pos[d]];
                found = 1;
            }
        }
        if (!found)
            break;
        uint16_t value = 0;
        int have = 0;
        for (int32_t d = num_deltas - 1; d >= 0; --d) {
            if (pos[d] < counts[d] && idxs[d][pos[d]] == smallest) {
                if (!have) {
                    value = vals[d][pos[d]];
                    have = 1;
                }
                ++pos[d];
            }
        }
        if (count < capacity) {
            out_idx[count] = smallest;
            out_val[count] = value;
        }
        ++count;
    }
    free(pos);
    return count;
}

/* ------------------------------------------------------------------ */
/* XXH64 integrity hash                                                */
/* ------------------------------------------------------------------ */

static const uint64_t XP1 = 11400714785074694791ULL;
static const uint64_t XP2 = 14029467366897019727ULL;
static const uint64_t XP3 = 1609587929392839161ULL;
static const uint64_t XP4 = 9650029242287828579ULL;
static const uint64_t XP5 = 2870177450012600261ULL;

static uint64_t rotl64(uint64_t x, int r) { return (x << r) | (x >> (64 - r)); }

static uint64_t read_le64(const uint8_t *p)
{
    uint64_t v = 0;
    for (int b = 7; b >= 0; --b)
        v = (v << 8) | p[b];
    return v;
}

static uint32_t read_le32(const uint8_t *p)
{
    return (uint32_t)p[0] | ((uint32_t)p[1] << 8) | ((uint32_t)p[2] << 16) |
           ((uint32_t)p[3] << 24);
}

static uint64_t xround(uint64_t acc, uint64_t lane)
{
    acc += lane * XP2;
    acc = rotl64(acc, 31);
    return acc * XP1;
}

/* XXH64 of `len` bytes at `data` with `seed`, step by step as the
 * specification gives it. */
uint64_t oracle_xxh64(const uint8_t *data, uint64_t len, uint64_t seed)
{
    const uint8_t *p = data;
    uint64_t left = len;
    uint64_t acc;
    if (len >= 32) {
        uint64_t a1 = seed + XP1 + XP2, a2 = seed + XP2, a3 = seed, a4 = seed - XP1;
        while (left >= 32) {
            a1 = xround(a1, read_le64(p));
            a2 = xround(a2, read_le64(p + 8));
            a3 = xround(a3, read_le64(p + 16));
            a4 = xround(a4, read_le64(p + 24));
            p += 32;
            left -= 32;
        }
        acc = rotl64(a1, 1) + rotl64(a2, 7) + rotl64(a3, 12) + rotl64(a4, 18);
        acc = (acc ^ xround(0, a1)) * XP1 + XP4;
        acc = (acc ^ xround(0, a2)) * XP1 + XP4;
        acc = (acc ^ xround(0, a3)) * XP1 + XP4;
        acc = (acc ^ xround(0, a4)) * XP1 + XP4;
    } else {
        acc = seed + XP5;
    }
    acc += len;
    while (left >= 8) {
        acc ^= xround(0, read_le64(p));
        acc = rotl64(acc, 27) * XP1 + XP4;
        p += 8;
        left -= 8;
    }
    if (left >= 4) {
        acc ^= (uint64_t)read_le32(p) * XP1;
        acc = rotl64(acc, 23) * XP2 + XP3;
        p += 4;
        left -= 4;
    }
    while (left >= 1) {
        acc ^= (uint64_t)(*p) * XP5;
        acc = rotl64(acc, 11) * XP1;
        ++p;
        --left;
    }
    acc ^= acc >> 33;
    acc *= XP2;
    acc ^= acc >> 29;
    acc *= XP3;
    acc ^= acc >> 32;
    return acc;
}

/* The hash of each `seg_bytes`-long piece of `data` (the last piece may be
 * shorter): the per-segment integrity check of Sec. 5.2. */
void oracle_hash_segments(const uint8_t *data, uint64_t len, uint64_t seg_bytes, uint64_t seed,
                          uint64_t *hashes)
{
    uint64_t s = 0;
    for (uint64_t off = 0; off < len; off += seg_bytes, ++s) {
        uint64_t n = len - off < seg_bytes ? len - off : seg_bytes;
        hashes[s] = oracle_xxh64(data + off, n, seed);
    }
}
