// Bimodal tensor runtime (paper section 7.2): which page set each tensor
// argument of a kernel uses, by tensor class and by the co-location state,
// and the moves between page sets when the state changes.
//
//  - Memory-bound best-effort weights keep two resident copies, one over
//    all channels and one over the best-effort channels; a kernel reads the
//    first while it runs alone (monopolization) and the second while
//    latency-sensitive kernels run beside it (colocation).  Nothing moves.
//  - Memory-bound latency-sensitive tensors have one copy, kept on the
//    latency-sensitive channels while best-effort work runs and moved to the
//    all-channel pool when it does not (a relayout on every state change).
//  - Intermediate results are written to the page set of the writing
//    kernel's state and read from where they were last written; their
//    buffers are reused through a free list.
//
// Host-only bookkeeping; moves are bimodal_relayout launches (a state
// change moves all latency-sensitive tensors in one batched relayout).
#include <algorithm>
#include <cstring>
#include <mutex>
#include <vector>

#include "host_common.hpp"

namespace sgdrc {

constexpr uint32_t kBmMagic = 0x424D4F44u;  // "BMOD"

struct BmTensor {
    uint32_t cls = 0;
    sgdrc_paged all{}, part{};
    uint64_t bytes = 0;      // size (weights, LS tensors) or capacity (activations)
    uint32_t shift = 0;
    int where = -1;          // SGDRC_BM_ALL, SGDRC_BM_PART, or -1 (no data yet)
    bool in_use = false;     // activations: acquired
};

struct Bimodal {
    uint32_t magic = kBmMagic;
    sgdrc_ctx *ctx = nullptr;
    int state = SGDRC_BM_MONOPOLY;
    std::mutex mu;
    std::vector<BmTensor> t;
};

static int check_bm(sgdrc_bimodal *bm, Bimodal **out)
{
    if (!bm)
        return set_error(SGDRC_EINVAL, "bimodal runtime is NULL");
    Bimodal *b = reinterpret_cast<Bimodal *>(bm);
    if (b->magic != kBmMagic)
        return set_error(SGDRC_EINVAL, "not a bimodal runtime");
    *out = b;
    return SGDRC_OK;
}

static int check_id(const Bimodal *b, uint32_t id)
{
    if (id >= b->t.size())
        return set_error(SGDRC_EINVAL, "tensor id %u not registered", id);
    return SGDRC_OK;
}

// Moves tensor x's data to page set ``to`` (relayout on ``stream``).
static int move_to(Bimodal *b, BmTensor &x, int to, void *stream)
{
    if (x.where == to)
        return SGDRC_OK;
    const sgdrc_paged *dst = to == SGDRC_BM_ALL ? &x.all : &x.part;
    const sgdrc_paged *src = to == SGDRC_BM_ALL ? &x.part : &x.all;
    const int rc = bimodal_relayout(b->ctx, dst, src, x.bytes, x.shift, stream);
    if (rc)
        return rc;
    x.where = to;
    return SGDRC_OK;
}

}  // namespace sgdrc

using namespace sgdrc;

extern "C" {

int sgdrc_bm_create(sgdrc_ctx *ctx, sgdrc_bimodal **out)
{
    clear_error();
    if (!out)
        return set_error(SGDRC_EINVAL, "out is NULL");
    if (ctx) {
        Ctx *c = nullptr;
        const int rc = check_ctx(ctx, &c);
        if (rc)
            return rc;
    }
    Bimodal *b = new (std::nothrow) Bimodal;
    if (!b)
        return set_error(SGDRC_ENOMEM, "out of host memory");
    b->ctx = ctx;
    *out = reinterpret_cast<sgdrc_bimodal *>(b);
    return SGDRC_OK;
}

int sgdrc_bm_destroy(sgdrc_bimodal *bm)
{
    clear_error();
    Bimodal *b = nullptr;
    const int rc = check_bm(bm, &b);
    if (rc)
        return rc;
    b->magic = 0;
    delete b;
    return SGDRC_OK;
}

int sgdrc_bm_register(sgdrc_bimodal *bm, uint32_t cls, const sgdrc_paged *all_form,
                      const sgdrc_paged *part_form, uint64_t n_bytes, uint32_t page_shift,
                      void *stream, uint32_t *id)
{
    clear_error();
    if (cls > SGDRC_BM_ACTIVATION)
        return set_error(SGDRC_EINVAL, "unknown tensor class %u", cls);
    int rc = check_shift(page_shift);
    if (rc)
        return rc;
    if ((rc = check_paged(all_form, "all_form")) || (rc = check_paged(part_form, "part_form")))
        return rc;
    if (n_bytes == 0 || !id)
        return set_error(SGDRC_EINVAL, "n_bytes is 0 or id is NULL");
    Bimodal *b = nullptr;
    if ((rc = check_bm(bm, &b)))
        return rc;
    std::lock_guard<std::mutex> lock(b->mu);
    if (cls != SGDRC_BM_ACTIVATION && !b->ctx)
        return set_error(SGDRC_ENODEV, "a runtime without a context holds activations only");
    BmTensor x;
    x.cls = cls;
    x.all = *all_form;
    x.part = *part_form;
    x.bytes = n_bytes;
    x.shift = page_shift;
    if (cls == SGDRC_BM_BE_WEIGHT) {
        // the second resident copy, over the best-effort channels
        x.where = SGDRC_BM_ALL;
        if ((rc = bimodal_relayout(b->ctx, &x.part, &x.all, n_bytes, page_shift, stream)))
            return rc;
    } else if (cls == SGDRC_BM_LS_TENSOR) {
        // data arrives in the all-channel form; it moves to the
        // latency-sensitive channels while best-effort work runs beside it
        x.where = SGDRC_BM_ALL;
        if (b->state == SGDRC_BM_COLOCATED && (rc = move_to(b, x, SGDRC_BM_PART, stream)))
            return rc;
    }
    b->t.push_back(x);
    *id = (uint32_t)(b->t.size() - 1);
    return SGDRC_OK;
}

int sgdrc_bm_set_state(sgdrc_bimodal *bm, int state, void *stream)
{
    clear_error();
    if (state != SGDRC_BM_MONOPOLY && state != SGDRC_BM_COLOCATED)
        return set_error(SGDRC_EINVAL, "unknown state %d", state);
    Bimodal *b = nullptr;
    int rc = check_bm(bm, &b);
    if (rc)
        return rc;
    std::lock_guard<std::mutex> lock(b->mu);
    if (state == b->state)
        return SGDRC_OK;
    // every latency-sensitive tensor moves to the new state's page set, all
    // in one batched relayout (one launch per 32 tensors)
    const int home = state == SGDRC_BM_COLOCATED ? SGDRC_BM_PART : SGDRC_BM_ALL;
    std::vector<sgdrc_relayout_item> moves;
    std::vector<BmTensor *> moved;
    for (BmTensor &x : b->t)
        if (x.cls == SGDRC_BM_LS_TENSOR && x.where != home) {
            sgdrc_relayout_item it{};
            it.dst = home == SGDRC_BM_ALL ? x.all : x.part;
            it.src = home == SGDRC_BM_ALL ? x.part : x.all;
            it.n_bytes = x.bytes;
            it.page_shift = x.shift;
            moves.push_back(it);
            moved.push_back(&x);
        }
    if (!moves.empty() &&
        (rc = bimodal_relayout_batch(b->ctx, moves.data(), (uint32_t)moves.size(), stream)))
        return rc;
    for (BmTensor *x : moved)
        x->where = home;
    b->state = state;
    return SGDRC_OK;
}

int sgdrc_bm_state(sgdrc_bimodal *bm, int *state)
{
    clear_error();
    if (!state)
        return set_error(SGDRC_EINVAL, "state is NULL");
    Bimodal *b = nullptr;
    const int rc = check_bm(bm, &b);
    if (rc)
        return rc;
    std::lock_guard<std::mutex> lock(b->mu);
    *state = b->state;
    return SGDRC_OK;
}

int sgdrc_bm_input(sgdrc_bimodal *bm, uint32_t id, sgdrc_paged *out, int *where)
{
    clear_error();
    if (!out)
        return set_error(SGDRC_EINVAL, "out is NULL");
    Bimodal *b = nullptr;
    int rc = check_bm(bm, &b);
    if (rc)
        return rc;
    std::lock_guard<std::mutex> lock(b->mu);
    if ((rc = check_id(b, id)))
        return rc;
    const BmTensor &x = b->t[id];
    int w = x.where;
    if (x.cls == SGDRC_BM_BE_WEIGHT)
        w = b->state == SGDRC_BM_COLOCATED ? SGDRC_BM_PART : SGDRC_BM_ALL;
    if (w < 0)
        return set_error(SGDRC_EINVAL, "tensor %u has not been written", id);
    *out = w == SGDRC_BM_ALL ? x.all : x.part;
    if (where)
        *where = w;
    return SGDRC_OK;
}

int sgdrc_bm_output(sgdrc_bimodal *bm, uint32_t id, sgdrc_paged *out, int *where)
{
    clear_error();
    if (!out)
        return set_error(SGDRC_EINVAL, "out is NULL");
    Bimodal *b = nullptr;
    int rc = check_bm(bm, &b);
    if (rc)
        return rc;
    std::lock_guard<std::mutex> lock(b->mu);
    if ((rc = check_id(b, id)))
        return rc;
    BmTensor &x = b->t[id];
    if (x.cls == SGDRC_BM_BE_WEIGHT)
        return set_error(SGDRC_EINVAL, "tensor %u is a weight (read-only)", id);
    if (x.cls == SGDRC_BM_ACTIVATION)
        x.where = b->state == SGDRC_BM_COLOCATED ? SGDRC_BM_PART : SGDRC_BM_ALL;
    *out = x.where == SGDRC_BM_ALL ? x.all : x.part;
    if (where)
        *where = x.where;
    return SGDRC_OK;
}

int sgdrc_bm_acquire(sgdrc_bimodal *bm, uint64_t n_bytes, uint32_t *id)
{
    clear_error();
    if (!id)
        return set_error(SGDRC_EINVAL, "id is NULL");
    Bimodal *b = nullptr;
    const int rc = check_bm(bm, &b);
    if (rc)
        return rc;
    std::lock_guard<std::mutex> lock(b->mu);
    int best = -1;
    for (size_t i = 0; i < b->t.size(); ++i) {
        const BmTensor &x = b->t[i];
        if (x.cls != SGDRC_BM_ACTIVATION || x.in_use || x.bytes < n_bytes)
            continue;
        if (best < 0 || x.bytes < b->t[best].bytes)
            best = (int)i;
    }
    if (best < 0)
        return set_error(SGDRC_ENOMEM, "no free activation buffer of %llu bytes",
                         (unsigned long long)n_bytes);
    b->t[best].in_use = true;
    b->t[best].where = -1;
    *id = (uint32_t)best;
    return SGDRC_OK;
}

int sgdrc_bm_release(sgdrc_bimodal *bm, uint32_t id)
{
    clear_error();
    Bimodal *b = nullptr;
    int rc = check_bm(bm, &b);
    if (rc)
        return rc;
    std::lock_guard<std::mutex> lock(b->mu);
    if ((rc = check_id(b, id)))
        return rc;
    BmTensor &x = b->t[id];
    if (x.cls != SGDRC_BM_ACTIVATION || !x.in_use)
        return set_error(SGDRC_EINVAL, "tensor %u is not an acquired activation", id);
    x.in_use = false;
    return SGDRC_OK;
}

}  // extern "C"
