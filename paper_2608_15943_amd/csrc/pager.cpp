// Host-side page allocator for paged KV storage.  A page is 64 positions of one
// sequence; the same page index is used in every producer's pool, so one table row per
// sequence serves all producers (they store the same positions, Eq. 3).  Sharing halves
// (or quarters) the producers, hence the bytes per page index, hence the pages a fixed
// amount of HBM holds: that is the capacity side of KV sharing.
//
// Pure host code: no device memory is touched; the caller copies table rows to the device.
#include <cstdint>
#include <vector>

#include "kvpipe.h"
#include "status.h"

using kvp::fail;
using kvp::ok;

struct kvp_pager {
    int n_pages, max_seqs, max_pages;
    std::vector<int32_t> table;   // [max_seqs][max_pages], -1 where unmapped
    std::vector<int32_t> held;    // pages held per sequence
    std::vector<int32_t> free;    // free pages; the back is handed out next
};

extern "C" int kvp_pager_create(int n_pages, int max_seqs, int max_pages_per_seq, kvp_pager** out) {
    if (!out) return fail(KVP_E_INVALID_ARG, "kvp_pager_create: NULL out");
    *out = nullptr;
    if (n_pages < 1 || max_seqs < 1 || max_pages_per_seq < 1)
        return fail(KVP_E_INVALID_ARG, "kvp_pager_create: sizes must be >= 1");
    if ((int64_t)max_seqs * max_pages_per_seq > (int64_t)1 << 31)
        return fail(KVP_E_INVALID_ARG, "kvp_pager_create: table of %d x %d entries is too large", max_seqs,
                    max_pages_per_seq);
    kvp_pager* p = new kvp_pager;
    p->n_pages = n_pages;
    p->max_seqs = max_seqs;
    p->max_pages = max_pages_per_seq;
    p->table.assign((size_t)max_seqs * max_pages_per_seq, -1);
    p->held.assign(max_seqs, 0);
    p->free.resize(n_pages);
    for (int i = 0; i < n_pages; ++i) p->free[i] = n_pages - 1 - i;   // page 0 first
    *out = p;
    return ok();
}

extern "C" void kvp_pager_destroy(kvp_pager* p) { delete p; }

extern "C" int kvp_pager_reserve(kvp_pager* p, int seq, int n_tokens) {
    if (!p) return fail(KVP_E_INVALID_ARG, "kvp_pager_reserve: NULL pager");
    if (seq < 0 || seq >= p->max_seqs) return fail(KVP_E_INVALID_ARG, "kvp_pager_reserve: sequence %d out of range", seq);
    if (n_tokens < 0) return fail(KVP_E_INVALID_ARG, "kvp_pager_reserve: n_tokens < 0");
    const int64_t need = ((int64_t)n_tokens + 63) / 64;
    if (need > p->max_pages)
        return fail(KVP_E_CAPACITY, "kvp_pager_reserve: %d tokens need %lld pages, a row holds %d", n_tokens,
                    (long long)need, p->max_pages);
    const int have = p->held[seq];
    if (need <= have) return ok();
    const int add = (int)need - have;
    if ((size_t)add > p->free.size())
        return fail(KVP_E_CAPACITY, "kvp_pager_reserve: %d more pages needed, %zu free", add, p->free.size());
    int32_t* row = p->table.data() + (size_t)seq * p->max_pages;
    for (int j = have; j < (int)need; ++j) {
        row[j] = p->free.back();
        p->free.pop_back();
    }
    p->held[seq] = (int)need;
    return ok();
}

extern "C" int kvp_pager_release(kvp_pager* p, int seq) {
    if (!p) return fail(KVP_E_INVALID_ARG, "kvp_pager_release: NULL pager");
    if (seq < 0 || seq >= p->max_seqs) return fail(KVP_E_INVALID_ARG, "kvp_pager_release: sequence %d out of range", seq);
    int32_t* row = p->table.data() + (size_t)seq * p->max_pages;
    for (int j = p->held[seq] - 1; j >= 0; --j) {   // the sequence's first page comes out first again
        p->free.push_back(row[j]);
        row[j] = -1;
    }
    p->held[seq] = 0;
    return ok();
}

extern "C" int kvp_pager_free_pages(const kvp_pager* p, int* n) {
    if (!p || !n) return fail(KVP_E_INVALID_ARG, "kvp_pager_free_pages: NULL argument");
    *n = (int)p->free.size();
    return ok();
}

extern "C" int kvp_pager_rows(const kvp_pager* p, const int32_t* seqs, int B, int32_t* out) {
    if (!p || !seqs || !out || B < 0) return fail(KVP_E_INVALID_ARG, "kvp_pager_rows: NULL argument or B < 0");
    for (int i = 0; i < B; ++i)
        if (seqs[i] < 0 || seqs[i] >= p->max_seqs)
            return fail(KVP_E_INVALID_ARG, "kvp_pager_rows: sequence %d out of range", seqs[i]);
    for (int i = 0; i < B; ++i) {
        const int32_t* row = p->table.data() + (size_t)seqs[i] * p->max_pages;
        for (int j = 0; j < p->max_pages; ++j) out[(size_t)i * p->max_pages + j] = row[j];
    }
    return ok();
}
