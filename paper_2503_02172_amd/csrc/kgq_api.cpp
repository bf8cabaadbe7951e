// C ABI of libkgq (declared in include/kgq.h): handle, parameter loading,
// argument validation, plan upload and the per-model stage sequence.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/kgq.h"
#include "kgq_internal.hpp"
#include "plan.hpp"

using namespace kgq;

namespace {

struct ParamSpec {
    int64_t rows, cols;     // element count = rows * cols
    bool entity;            // takes cfg.entity_dtype
};

struct DevBuf {
    void* p = nullptr;
    size_t bytes = 0;
};

struct ProfPair {
    int stage;
    hipEvent_t start, stop;
};

// Scratch of one execute in flight. A handle owns cfg.concurrency lanes;
// consecutive executes use them round-robin, and an execute's stream first
// waits (on the device) for the lane's previous use to finish.
struct Lane {
    float* states = nullptr;
    float* xbuf = nullptr;        // BetaE MLP input / intersection input
    float* h1 = nullptr;
    float* h2 = nullptr;
    float* logits = nullptr;
    float* zfeat = nullptr;
    float* zmean = nullptr;
    float* gate = nullptr;
    float* qpack = nullptr;
    double* cq = nullptr;
    float* scores = nullptr;
    float* gemm_ws = nullptr;     // split-K partials of small dense layers
    int64_t gemm_ws_elems = 0;
    float* score_ws = nullptr;    // split-d partials of the VALU scorers at small batches
    int64_t score_ws_elems = 0;
    int32_t* cand_idx[2] = {nullptr, nullptr};   // top-k candidates of long rows
    float* cand_score[2] = {nullptr, nullptr};
    uint32_t* chunk_key = nullptr;   // the scorer's chunk keys for top-k [rows x ceil(N / 64)]
    int* dflag = nullptr;
    int* hflag = nullptr;         // pinned
    // plan images: per-structure cache slots + a ring of two for mixed batches
    int32_t* plan_dev = nullptr;  // (kNumStructures + 2) slots
    int32_t* plan_host = nullptr; // pinned staging, same slot layout
    hipEvent_t slot_event[kNumStructures + 2]{};
    bool slot_event_live[kNumStructures + 2]{};
    int cached_B[kNumStructures];
    std::unique_ptr<Plan> cached_plan[kNumStructures];
    int ring_next = 0;
    hipEvent_t done = nullptr;    // recorded after the lane's last execute
    bool done_live = false;
    Lane() { for (int i = 0; i < kNumStructures; ++i) cached_B[i] = -1; }
};

thread_local std::string g_create_error;

std::mutex g_scratch_mu;
std::map<int, unsigned char*> g_scratch_addr;   // device ordinal -> address of `scratch`

}  // namespace

// Device scratch of kgq_execute_mixed_noalloc: one array per GPU, in the
// library's code object, held until the process ends. In host code the name
// `scratch` is only a stand-in; its device address on each GPU comes from
// hipGetSymbolAddress (taken once per device, with that device current) and
// is the only form host code passes on.
static __device__ __align__(256) unsigned char scratch[KGQ_NOALLOC_SCRATCH_BYTES];

struct kgq_handle {
    kgq_config cfg{};
    bool dry = false;
    bool checked = false;
    std::string err;

    std::map<std::string, ParamSpec> specs;
    std::map<std::string, bool> loaded;
    std::map<std::string, float*> dparam;   // device fp32 parameters (weights, relations)

    // derived entity tables
    int64_t n_blocks = 0;
    float* ent_rm = nullptr;      // GQE/Q2B [N x d]; BetaE alpha|beta, ConE [axis; 0], LogicE [l; u] [N x 2d]
    float* ent_blk = nullptr;     // scoring table: GQE/Q2B/LogicE blocked points; BetaE row-major U|V;
                                  // ConE blocked half-angle sin | cos
    double* ent_const = nullptr;  // BetaE E_e [n_pad]
    uint16_t* ent_planes = nullptr;   // BetaE [U | V] rows of ent_blk as three bf16 planes (when 2d % 32 == 0)
    float* rel_o_sp = nullptr;    // Q2B softplus(offset_raw) [R x d]
    float cone_modulus = 0.f;     // ConE distance scale (host copy of "modulus")
    float* int_cat_w = nullptr;   // ConE [inter.axis.w1; inter.arg.w1] [2d x 2d]
    float* int_cat_b = nullptr;   // ConE [inter.axis.b1; inter.arg.b1] [2d]
    // BetaE, ConE, LogicE: the first projection layer is linear in its
    // input (the source state plus or next to Rel[r]), so for first-hop
    // projections (input = an anchor entity) it splits into two
    // parameter-only tables, built when their inputs are loaded:
    float* proj1_ent = nullptr;   // [N x 4d]  entity state . W1^T (LogicE: its state columns of W1)
    float* proj1_rel = nullptr;   // [R x 4d]  Rel . W1^T + b1 (LogicE: its relation columns)
    bool proj1_ready = false;
    // dense-layer weights split into three bf16 planes each (weight -> planes),
    // for the FP32-accurate bf16 matrix-core GEMM; the split is redone when a
    // weight is loaded
    std::map<const float*, uint16_t*> wplanes;
    int dense_path = KGQ_DENSE_AUTO;

    // structure id -> compiled program: the built-ins for this model, then
    // the structures compiled on this handle
    std::vector<const Program*> table;
    std::vector<std::unique_ptr<Program>> compiled;

    // scratch lanes (each sized for max_batch at create): executes on
    // different lanes may run concurrently on different streams
    std::vector<std::unique_ptr<Lane>> lanes;
    int next_lane = 0;
    int64_t plan_words = 0;
    // what one lane holds: state rows, rows of one dense-layer level or
    // intersection stage, groups of one intersection stage, scored rows
    int64_t cap_rows = 0, cap_mlp = 0, cap_groups = 0, cap_score_rows = 0;

    // the device address of the static scratch array on this handle's GPU
    // (kgq_execute_mixed_noalloc), taken at create
    unsigned char* noalloc_scratch = nullptr;

    std::vector<void*> allocations;
    int64_t bytes_total = 0;      // device bytes allocated by the handle
    int64_t bytes_params = 0;     // ... of which parameters and derived tables

    // profiling
    int prof = 0;                 // bitmask of stages being timed
    std::vector<ProfPair> prof_pending;
    std::vector<hipEvent_t> prof_pool;
    double prof_ms[KGQ_NUM_STAGES]{};
    int64_t prof_n[KGQ_NUM_STAGES]{};
    hipEvent_t prof_ref = nullptr;                     // time origin of the intervals
    std::vector<double> prof_iv[KGQ_NUM_STAGES];       // (start, end) ms pairs
};

namespace {

kgq_status fail(kgq_handle* h, kgq_status s, const std::string& msg)
{
    if (h) h->err = msg;
    return s;
}

#define HIP_TRY(h, call)                                                                   \
    do {                                                                                   \
        hipError_t e_ = (call);                                                            \
        if (e_ != hipSuccess)                                                              \
            return fail((h), e_ == hipErrorOutOfMemory ? KGQ_E_OOM : KGQ_E_DEVICE,         \
                        std::string(#call) + ": " + hipGetErrorString(e_));                 \
    } while (0)

void build_specs(kgq_handle* h)
{
    const int64_t N = h->cfg.n_entities, R = h->cfg.n_relations, d = h->cfg.dim;
    auto& s = h->specs;
    switch (h->cfg.model) {
    case KGQ_GQE:
        s["entity"] = {N, d, true};
        s["relation"] = {R, d, false};
        s["inter.w1"] = {d, d, false};
        s["inter.b1"] = {1, d, false};
        s["inter.w2"] = {d, d, false};
        s["inter.b2"] = {1, d, false};
        break;
    case KGQ_Q2B:
        s["entity"] = {N, d, true};
        s["relation.center"] = {R, d, false};
        s["relation.offset_raw"] = {R, d, false};
        for (const char* grp : {"inter.center.", "inter.offset."}) {
            s[std::string(grp) + "w1"] = {d, d, false};
            s[std::string(grp) + "b1"] = {1, d, false};
            s[std::string(grp) + "w2"] = {d, d, false};
            s[std::string(grp) + "b2"] = {1, d, false};
        }
        break;
    case KGQ_CONE:
        s["entity.axis"] = {N, d, true};
        s["relation"] = {R, 2 * d, false};
        s["proj.w1"] = {4 * d, 2 * d, false};
        s["proj.b1"] = {1, 4 * d, false};
        s["proj.w2"] = {4 * d, 4 * d, false};
        s["proj.b2"] = {1, 4 * d, false};
        s["proj.w3"] = {2 * d, 4 * d, false};
        s["proj.b3"] = {1, 2 * d, false};
        for (const char* grp : {"inter.axis.", "inter.arg."}) {
            s[std::string(grp) + "w1"] = {d, 2 * d, false};
            s[std::string(grp) + "b1"] = {1, d, false};
            s[std::string(grp) + "w2"] = {d, d, false};
            s[std::string(grp) + "b2"] = {1, d, false};
        }
        s["modulus"] = {1, 1, false};
        break;
    case KGQ_LOGICE:
        s["entity.bounds"] = {N, 2 * d, true};
        s["relation"] = {R, d, false};
        s["proj.w1"] = {4 * d, 3 * d, false};
        s["proj.b1"] = {1, 4 * d, false};
        s["proj.w2"] = {4 * d, 4 * d, false};
        s["proj.b2"] = {1, 4 * d, false};
        s["proj.w3"] = {2 * d, 4 * d, false};
        s["proj.b3"] = {1, 2 * d, false};
        break;
    default:
        s["entity.alpha_beta"] = {N, 2 * d, true};
        s["relation"] = {R, 2 * d, false};
        s["proj.w1"] = {4 * d, 2 * d, false};
        s["proj.b1"] = {1, 4 * d, false};
        s["proj.w2"] = {4 * d, 4 * d, false};
        s["proj.b2"] = {1, 4 * d, false};
        s["proj.w3"] = {2 * d, 4 * d, false};
        s["proj.b3"] = {1, 2 * d, false};
        s["inter.w1"] = {2 * d, 2 * d, false};
        s["inter.b1"] = {1, 2 * d, false};
        s["inter.w2"] = {d, 2 * d, false};
        s["inter.b2"] = {1, d, false};
        break;
    }
    for (auto& kv : s) h->loaded[kv.first] = false;
}

// Structure table and the capacities of one lane (also for a
// validation-only handle, which allocates nothing).
void build_table(kgq_handle* h)
{
    const kgq_config& c = h->cfg;
    const int64_t Bm = c.max_batch;
    int words = 64;   // plan-image words per query: room for structures larger than the built-ins
    for (int id = 0; id < kNumStructures; ++id) {
        const Program* g = builtin_program(c.model, id);
        h->table.push_back(g);
        if (g->supported) words = std::max(words, g->image_words);
    }
    // slots start at 16-byte boundaries (the upload kernel moves 16-byte words)
    h->plan_words = (Bm * words + kPlanOverheadWords + 3) / 4 * 4;
    h->cap_rows = Bm * kStateRowsPerQuery;
    h->cap_mlp = 3 * Bm;
    h->cap_groups = h->cap_mlp / 2;   // a group has at least two inputs
    const int tq = score_row_pad(c.model);
    h->cap_score_rows = ((2 * Bm + tq - 1) / tq) * tq;
}

// Largest batch of one structure that a lane holds.
int64_t max_batch_for(const kgq_handle* h, const Program& g)
{
    int64_t mb = h->cfg.max_batch;
    mb = std::min<int64_t>(mb, h->cap_rows / std::max<int64_t>(1, (int64_t)g.ops.size()));
    if (g.max_stage_level) mb = std::min<int64_t>(mb, h->cap_mlp / g.max_stage_level);
    if (g.max_stage_inputs) mb = std::min<int64_t>(mb, h->cap_mlp / g.max_stage_inputs);
    if (g.max_stage_groups) mb = std::min<int64_t>(mb, h->cap_groups / g.max_stage_groups);
    mb = std::min<int64_t>(mb, h->cap_score_rows / (int64_t)g.answer.size());
    mb = std::min<int64_t>(mb, (h->plan_words - kPlanOverheadWords) / g.image_words);
    return mb;
}

const Program* program_of(const kgq_handle* h, int id)
{
    return (id >= 0 && id < (int)h->table.size()) ? h->table[id] : nullptr;
}

kgq_status dev_alloc(kgq_handle* h, void** p, size_t bytes)
{
    *p = nullptr;
    if (bytes == 0) bytes = 16;
    hipError_t e = hipMalloc(p, bytes);
    if (e != hipSuccess) {
        *p = nullptr;
        return fail(h, e == hipErrorOutOfMemory ? KGQ_E_OOM : KGQ_E_DEVICE,
                    std::string("hipMalloc(") + std::to_string(bytes) + "): " + hipGetErrorString(e));
    }
    h->allocations.push_back(*p);
    h->bytes_total += (int64_t)bytes;
    return KGQ_OK;
}

template <typename T>
kgq_status dev_alloc_t(kgq_handle* h, T** p, size_t count)
{
    void* v = nullptr;
    kgq_status s = dev_alloc(h, &v, count * sizeof(T));
    *p = reinterpret_cast<T*>(v);
    return s;
}

void free_all(kgq_handle* h)
{
    if (h->dry) return;
    // Teardown: errors are ignored, every resource is released regardless.
    (void)hipSetDevice(h->cfg.device);
    (void)hipDeviceSynchronize();
    for (void* p : h->allocations) (void)hipFree(p);
    h->allocations.clear();
    for (auto& L : h->lanes) {
        if (L->hflag) (void)hipHostFree(L->hflag);
        if (L->plan_host) (void)hipHostFree(L->plan_host);
        for (int i = 0; i < kNumStructures + 2; ++i)
            if (L->slot_event[i]) (void)hipEventDestroy(L->slot_event[i]);
        if (L->done) (void)hipEventDestroy(L->done);
    }
    h->lanes.clear();
    for (auto& pp : h->prof_pending) {
        (void)hipEventDestroy(pp.start);
        (void)hipEventDestroy(pp.stop);
    }
    for (hipEvent_t e : h->prof_pool) (void)hipEventDestroy(e);
    if (h->prof_ref) (void)hipEventDestroy(h->prof_ref);
}

// Floats of one scored row in the packed query buffer: GQE d; Query2Box
// (center, offset), BetaE (alpha, beta) and LogicE (l, u) 2d; ConE 4d (the
// half-angle cosine and sine of axis and aperture).
int64_t qpack_row_floats(int model, int d)
{
    return (int64_t)d * (model == KGQ_GQE ? 1 : model == KGQ_CONE ? 4 : 2);
}

kgq_status allocate_all(kgq_handle* h)
{
    const kgq_config& c = h->cfg;
    const int64_t N = c.n_entities, d = c.dim, Bm = c.max_batch;
    const int W = (c.model == KGQ_GQE) ? (int)d : (int)(2 * d);
    h->n_blocks = (N + kEntBlock - 1) / kEntBlock;
    const int64_t n_pad = h->n_blocks * kEntBlock;
    kgq_status s;
#define ALLOC(ptr, count) if ((s = dev_alloc_t(h, &(ptr), (size_t)(count))) != KGQ_OK) return s
    // parameters other than the entity table
    for (auto& kv : h->specs) {
        if (kv.second.entity) continue;
        float* p = nullptr;
        ALLOC(p, kv.second.rows * kv.second.cols);
        h->dparam[kv.first] = p;
    }
    if (mlp_model(c.model)) {
        ALLOC(h->ent_rm, N * 2 * d);
        ALLOC(h->ent_blk, n_pad * 2 * d);
        if (c.model == KGQ_BETAE) ALLOC(h->ent_const, n_pad);
        if (c.model == KGQ_BETAE && (2 * d) % 32 == 0) ALLOC(h->ent_planes, 3 * n_pad * 2 * d);
        ALLOC(h->proj1_ent, N * 4 * d);
        ALLOC(h->proj1_rel, (int64_t)c.n_relations * 4 * d);
        if (c.model == KGQ_CONE) {
            ALLOC(h->int_cat_w, 4 * d * d);
            ALLOC(h->int_cat_b, 2 * d);
        }
    } else {
        ALLOC(h->ent_rm, N * d);
        ALLOC(h->ent_blk, n_pad * d);
        if (c.model == KGQ_Q2B) ALLOC(h->rel_o_sp, (int64_t)c.n_relations * d);
    }
    // bf16 planes of every dense-layer weight whose K (its columns) the
    // bf16 matrix-core GEMM takes, rows padded to whole 32-wide stages
    for (auto& kv : h->specs) {
        const std::string& n = kv.first;
        const bool weight = n.size() > 3 && n[n.size() - 3] == '.' && n[n.size() - 2] == 'w' &&
                            n.back() >= '1' && n.back() <= '3';
        if (kv.second.entity || !weight || kv.second.cols % 4 != 0 || kv.second.cols < 32) continue;
        uint16_t* planes = nullptr;
        ALLOC(planes, 3 * kv.second.rows * plane_ld(kv.second.cols));
        h->wplanes[h->dparam.at(n)] = planes;
    }
    if (h->int_cat_w && (2 * d) % 4 == 0 && 2 * d >= 32) {
        uint16_t* planes = nullptr;
        ALLOC(planes, 3 * 2 * d * plane_ld(2 * d));
        h->wplanes[h->int_cat_w] = planes;
    }
    h->bytes_params = h->bytes_total;   // everything after this is execute scratch
    const int n_lanes = c.concurrency > 0 ? c.concurrency : 1;
    for (int li = 0; li < n_lanes; ++li) {
        h->lanes.emplace_back(new Lane());
        Lane& L = *h->lanes.back();
        ALLOC(L.states, h->cap_rows * W);
        const int64_t m_max = h->cap_mlp;   // rows of one MLP level / intersection stage inputs
        if (mlp_model(c.model)) {
            ALLOC(L.xbuf, m_max * (c.model == KGQ_LOGICE ? 3 : 2) * d);
            ALLOC(L.h1, m_max * 4 * d);
            ALLOC(L.h2, m_max * 4 * d);
            if (c.model == KGQ_CONE) {
                ALLOC(L.zmean, h->cap_groups * d);
                ALLOC(L.gate, h->cap_groups * d);
            }
        } else {
            ALLOC(L.h1, m_max * d);
            if (c.model == KGQ_Q2B) {
                ALLOC(L.zfeat, m_max * d);
                ALLOC(L.zmean, h->cap_groups * d);
                ALLOC(L.gate, h->cap_groups * d);
            }
        }
        ALLOC(L.logits, m_max * d);
        ALLOC(L.qpack, h->cap_score_rows * qpack_row_floats(c.model, (int)d));
        ALLOC(L.cq, h->cap_score_rows);
        ALLOC(L.scores, Bm * N);
        // split-K runs only while a layer has fewer than 128 output tiles of
        // 64 x 64, so 16 slices of it stay below 16 x 128 x 4096 floats
        {
            const int64_t n_max = mlp_model(c.model) ? 4 * d : d;
            L.gemm_ws_elems = std::min<int64_t>(16 * 3 * Bm * n_max, (int64_t)16 * 128 * 4096);
            ALLOC(L.gemm_ws, L.gemm_ws_elems);
        }
        if (c.model != KGQ_BETAE) {
            // 16 slices x 2 fields x the padded rows of a small batch x the
            // padded entities, at most 8 Mi floats (fewer slices if tight)
            L.score_ws_elems = std::min<int64_t>(16 * 2 * (2 * Bm + 64) * n_pad, (int64_t)8 << 20);
            ALLOC(L.score_ws, L.score_ws_elems);
        }
        const int64_t ncand = topk_scratch_elems(Bm, N, kMaxK);
        for (int i = 0; i < 2; ++i) {
            ALLOC(L.cand_idx[i], ncand);
            ALLOC(L.cand_score[i], ncand);
        }
        ALLOC(L.chunk_key, Bm * ((N + kKeyChunk - 1) / kKeyChunk));
        ALLOC(L.dflag, 1);
        ALLOC(L.plan_dev, (int64_t)(kNumStructures + 2) * h->plan_words);
        hipError_t e = hipHostMalloc((void**)&L.hflag, sizeof(int), hipHostMallocDefault);
        if (e != hipSuccess) return fail(h, KGQ_E_OOM, "hipHostMalloc(flag)");
        // coherent: the upload kernel reads it over the bus, and a slot is
        // rewritten by the host after earlier reads, so no stale copy may
        // stay in a device cache
        e = hipHostMalloc((void**)&L.plan_host, sizeof(int32_t) * (kNumStructures + 2) * h->plan_words,
                          hipHostMallocCoherent);
        if (e != hipSuccess) return fail(h, KGQ_E_OOM, "hipHostMalloc(plan staging)");
        for (int i = 0; i < kNumStructures + 2; ++i)
            HIP_TRY(h, hipEventCreateWithFlags(&L.slot_event[i], hipEventDisableTiming));
        HIP_TRY(h, hipEventCreateWithFlags(&L.done, hipEventDisableTiming));
        HIP_TRY(h, hipMemset(L.dflag, 0, sizeof(int)));
    }
#undef ALLOC
    return KGQ_OK;
}

// --- profiling -------------------------------------------------------------

hipEvent_t prof_event(kgq_handle* h)
{
    if (!h->prof_pool.empty()) {
        hipEvent_t e = h->prof_pool.back();
        h->prof_pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

struct StageTimer {
    kgq_handle* h;
    int stage;
    hipStream_t s;
    hipEvent_t a = nullptr, b = nullptr;
    StageTimer(kgq_handle* h_, int st, hipStream_t s_) : h(h_), stage(st), s(s_)
    {
        if ((h->prof >> stage) & 1) {
            a = prof_event(h);
            b = prof_event(h);
            if (!a || !b || hipEventRecord(a, s) != hipSuccess) {
                // no timing for this stage: hand the events back to the pool
                if (a) h->prof_pool.push_back(a);
                if (b) h->prof_pool.push_back(b);
                a = b = nullptr;
            }
        }
    }
    ~StageTimer()
    {
        if (!a) return;
        if (hipEventRecord(b, s) == hipSuccess) {
            h->prof_pending.push_back({stage, a, b});
        } else {
            h->prof_pool.push_back(a);
            h->prof_pool.push_back(b);
        }
    }
};

void prof_collect(kgq_handle* h)
{
    for (auto& pp : h->prof_pending) {
        float ms = 0.f, t0 = 0.f, t1 = 0.f;
        if (hipEventSynchronize(pp.stop) == hipSuccess && hipEventElapsedTime(&ms, pp.start, pp.stop) == hipSuccess) {
            h->prof_ms[pp.stage] += ms;
            h->prof_n[pp.stage] += 1;
            if (h->prof_ref && hipEventElapsedTime(&t0, h->prof_ref, pp.start) == hipSuccess &&
                hipEventElapsedTime(&t1, h->prof_ref, pp.stop) == hipSuccess) {
                h->prof_iv[pp.stage].push_back(t0);
                h->prof_iv[pp.stage].push_back(t1);
            }
        }
        h->prof_pool.push_back(pp.start);
        h->prof_pool.push_back(pp.stop);
    }
    h->prof_pending.clear();
}

// --- execute helpers ----------------------------------------------------------

bool all_loaded(const kgq_handle* h, std::string& missing)
{
    for (auto& kv : h->loaded)
        if (!kv.second) {
            missing = kv.first;
            return false;
        }
    return true;
}

kgq_status check_outputs(kgq_handle* h, int32_t batch, const void* anchors, const void* rels, int32_t k,
                         const float* out_scores, const int32_t* out_idx, const float* out_score)
{
    if (batch < 1 || batch > h->cfg.max_batch)
        return fail(h, KGQ_E_INVALID_ARG, "batch " + std::to_string(batch) + " outside [1, max_batch=" +
                                              std::to_string(h->cfg.max_batch) + "]");
    if (!anchors || !rels) return fail(h, KGQ_E_INVALID_ARG, "anchors and relations must not be NULL");
    if ((out_idx == nullptr) != (out_score == nullptr))
        return fail(h, KGQ_E_INVALID_ARG, "out_topk_idx and out_topk_score must both be set or both be NULL");
    if (!out_scores && !out_idx) return fail(h, KGQ_E_INVALID_ARG, "no output requested");
    if (out_idx) {
        const int64_t kmax = h->cfg.n_entities < kMaxK ? h->cfg.n_entities : kMaxK;
        if (k < 1 || k > kmax)
            return fail(h, KGQ_E_INVALID_ARG, "k=" + std::to_string(k) + " outside [1, " + std::to_string(kmax) + "]");
    }
    std::string missing;
    if (!all_loaded(h, missing)) return fail(h, KGQ_E_NOT_LOADED, "parameter '" + missing + "' not loaded");
    return KGQ_OK;
}

// A lowered batch must fit the lane's scratch.
kgq_status check_capacity(kgq_handle* h, const Plan& p)
{
    const int tq = score_row_pad(h->cfg.model);
    const int64_t srows = ((int64_t)(p.n_score_rows + tq - 1) / tq) * tq;
    const char* what = nullptr;
    if (p.n_state_rows > h->cap_rows) what = "state rows";
    else if (p.max_level > h->cap_mlp || p.max_and_in > h->cap_mlp) what = "dense-layer rows";
    else if (p.max_and_groups > h->cap_groups) what = "intersection groups";
    else if (srows > h->cap_score_rows) what = "scored rows";
    else if ((int64_t)p.image.size() > h->plan_words) what = "plan words";
    if (!what) return KGQ_OK;
    return fail(h, KGQ_E_INVALID_ARG,
                std::string("the batch needs more ") + what + " than the handle's scratch (sized for max_batch=" +
                    std::to_string(h->cfg.max_batch) +
                    " built-in queries) holds; split it (kgq_structure_info gives the largest batch of one "
                    "structure)");
}

// Upload a plan image into device slot `slot` (after the slot's last use:
// the host waits for the execute that last read the slot, which also retires
// the previous upload out of the slot's pinned staging). The upload is a
// kernel in the caller's stream that reads the pinned staging over the bus:
// an asynchronous copy there goes through a copy engine and costs about
// 26 us of idle device between the previous execute's kernels and this
// one's, a copy on a stream of its own still about 15 us of cross-queue wait.
kgq_status upload_plan(kgq_handle* h, Lane& L, const Plan& p, int slot, hipStream_t s, int32_t* dst = nullptr)
{
    if ((int64_t)p.image.size() > h->plan_words) return fail(h, KGQ_E_DEVICE, "plan image exceeds its slot");
    if (L.slot_event_live[slot]) HIP_TRY(h, hipEventSynchronize(L.slot_event[slot]));
    int32_t* host = L.plan_host + (int64_t)slot * h->plan_words;
    std::memcpy(host, p.image.data(), p.image.size() * sizeof(int32_t));
    if (!dst) dst = L.plan_dev + (int64_t)slot * h->plan_words;
    launch_fetch_words(host, dst, (int64_t)p.image.size(), s);
    return KGQ_OK;
}

// Next scratch lane, round-robin. The caller's stream waits (on the device)
// until the lane's previous execute, possibly on another stream, is done.
kgq_status acquire_lane(kgq_handle* h, hipStream_t s, Lane** out)
{
    Lane* L = h->lanes[h->next_lane].get();
    h->next_lane = (h->next_lane + 1) % (int)h->lanes.size();
    if (L->done_live) HIP_TRY(h, hipStreamWaitEvent(s, L->done, 0));
    *out = L;
    return KGQ_OK;
}

kgq_status run_plan(kgq_handle* h, Lane& L, const Plan& p, const int32_t* P, const int32_t* anchors,
                    const int32_t* rels, int sa, int sr, int fixed_na, int fixed_nr, bool mixed, int32_t k,
                    float* out_scores, int32_t* out_idx, float* out_score, hipStream_t s)
{
    const kgq_config& c = h->cfg;
    const int d = c.dim;
    const int W = (c.model == KGQ_GQE) ? d : 2 * d;
    const int64_t N = c.n_entities;
    const int n_rel = c.n_relations;
    auto param = [&](const char* n) { return h->dparam.at(n); };
    // dense layers of this execute may split K over the lane's workspace
    auto gemm = [&](GemmArgs g) {
        g.ws = L.gemm_ws;
        g.ws_elems = L.gemm_ws_elems;
        if (h->dense_path != KGQ_DENSE_FP32) {
            auto pl = h->wplanes.find(g.W);
            if (pl != h->wplanes.end()) g.Wp = pl->second;
            g.bf16x3_always = h->dense_path == KGQ_DENSE_BF16X3;
        }
        launch_gemm(g, s);
    };

    if (h->checked) {
        launch_clear_flag(L.dflag, s);
        launch_validate(anchors, rels, mixed ? P + p.off_arity : nullptr, p.B, sa, sr, fixed_na, fixed_nr,
                        N, n_rel, L.dflag, s);
    }
    const bool betae = c.model == KGQ_BETAE, q2b = c.model == KGQ_Q2B;
    const bool cone = c.model == KGQ_CONE, logice = c.model == KGQ_LOGICE;
    const bool mlp = mlp_model(c.model);
    const float* rel_c = q2b ? param("relation.center") : c.model == KGQ_GQE ? param("relation") : nullptr;
    const float* rel_ab = mlp ? param("relation") : nullptr;
    const std::string pre = q2b ? "inter.center." : "inter.";

    for (const Stage& st : p.stages) {
        if (st.kind == ST_CHAIN) {
            // GQE / Query2Box: every translation chain of the batch
            StageTimer t(h, 0, s);
            launch_chain(c.model, P + st.a, P + st.b, P + st.c, P + st.d, st.count, anchors, rels, h->ent_rm, rel_c,
                         h->rel_o_sp, N, n_rel, d, L.states, L.dflag, s);
        } else if (st.kind == ST_LEVEL) {
            // BetaE, ConE, LogicE: one projection MLP pass over every
            // projection at this stage and hop
            const int M = st.count;
            const int in_w = logice ? 3 * d : 2 * d;   // LogicE concatenates Rel[r] to the state
            if (st.table) {
                // first hop from the anchors: the first layer is a gather
                // from the precomputed tables
                StageTimer t(h, 0, s);
                launch_betae_proj1(P + st.b, P + st.c, M, anchors, rels, h->proj1_ent, h->proj1_rel, N, n_rel, 4 * d,
                                   L.h1, L.dflag, s);
            } else {
                {
                    StageTimer t(h, 0, s);
                    if (betae)
                        launch_betae_proj_prep(P + st.a, P + st.b, P + st.c, P + st.d, M, anchors, rels, L.states,
                                               h->ent_rm, rel_ab, N, n_rel, d, L.xbuf, L.dflag, s);
                    else
                        launch_mlp_proj_prep(c.model, P + st.a, P + st.b, P + st.c, P + st.d, M, anchors, rels,
                                             L.states, h->ent_rm, rel_ab, N, n_rel, d, L.xbuf, L.dflag, s);
                }
                StageTimer t(h, 1, s);
                gemm({L.xbuf, in_w, param("proj.w1"), in_w, param("proj.b1"), L.h1, 4 * d, nullptr, M, 4 * d, in_w,
                      EPI_RELU});
            }
            {
                StageTimer t(h, 1, s);
                gemm({L.h1, 4 * d, param("proj.w2"), 4 * d, param("proj.b2"), L.h2, 4 * d, nullptr, M, 4 * d, 4 * d,
                      EPI_RELU});
            }
            // the last layer writes the model's output map through the row map
            GemmArgs g3{L.h2, 4 * d, param("proj.w3"), 4 * d, param("proj.b3"), L.states, 2 * d, P + st.e, M, 2 * d,
                        4 * d, betae ? EPI_BETA_REG : cone ? EPI_CONE_ANGLES : EPI_SIGMOID};
            g3.epi_split = d;
            {
                StageTimer t(h, 1, s);
                gemm(g3);
            }
            if (logice) {
                StageTimer t(h, 0, s);
                launch_logic_bounds(P + st.e, M, d, L.states, s);
            }
        } else {
            // every intersection group of one stage; its inputs are the rows
            // in_base .. in_base + n_in - 1 of the state buffer
            GroupArgs g{P + st.a, P + st.b, P + st.c, P + st.d, P + st.e, P + st.f, st.count};
            const float* sin = L.states + (int64_t)st.in_base * W;
            const int n_in = st.n_in;
            if (logice) {
                StageTimer t(h, 2, s);
                launch_logic_combine(c.tnorm, g, sin, d, L.states, s);
                continue;
            }
            if (cone) {
                {
                    StageTimer t(h, 2, s);
                    launch_cone_int_prep(g, sin, d, L.xbuf, s);
                }
                {
                    // both set functions' first layers, stacked: [attention | aperture] hidden
                    StageTimer t(h, 1, s);
                    gemm({L.xbuf, 2 * d, h->int_cat_w, 2 * d, h->int_cat_b, L.h1, 2 * d, nullptr, n_in, 2 * d, 2 * d,
                          EPI_RELU});
                }
                {
                    StageTimer t(h, 1, s);
                    gemm({L.h1, 2 * d, param("inter.axis.w2"), d, param("inter.axis.b2"), L.logits, d, nullptr, n_in,
                          d, d, EPI_NONE});
                }
                {
                    StageTimer t(h, 2, s);
                    launch_cone_combine_axis(g, sin, L.logits, L.h1, d, L.zmean, L.states, s);
                }
                {
                    StageTimer t(h, 1, s);
                    gemm({L.zmean, d, param("inter.arg.w2"), d, param("inter.arg.b2"), L.gate, d, nullptr, st.count,
                          d, d, EPI_NONE});
                }
                StageTimer t(h, 2, s);
                launch_cone_combine_arg(g, sin, L.gate, d, L.states, s);
                continue;
            }
            if (betae) {
                {
                    StageTimer t(h, 2, s);
                    launch_betae_int_prep(g, sin, d, L.xbuf, s);
                }
                {
                    StageTimer t(h, 1, s);
                    gemm({L.xbuf, 2 * d, param("inter.w1"), 2 * d, param("inter.b1"), L.h1, 2 * d, nullptr, n_in,
                          2 * d, 2 * d, EPI_RELU});
                }
                {
                    StageTimer t(h, 1, s);
                    gemm({L.h1, 2 * d, param("inter.w2"), 2 * d, param("inter.b2"), L.logits, d, nullptr, n_in, d,
                          2 * d, EPI_NONE});
                }
                StageTimer t(h, 2, s);
                launch_betae_combine(g, L.xbuf, L.logits, d, L.states, s);
                continue;
            }
            {
                StageTimer t(h, 1, s);
                gemm({sin, W, param((pre + "w1").c_str()), d, param((pre + "b1").c_str()), L.h1, d, nullptr, n_in, d,
                      d, EPI_RELU});
            }
            {
                StageTimer t(h, 1, s);
                gemm({L.h1, d, param((pre + "w2").c_str()), d, param((pre + "b2").c_str()), L.logits, d, nullptr,
                      n_in, d, d, EPI_NONE});
            }
            if (q2b) {
                StageTimer t(h, 1, s);
                gemm({sin + d, W, param("inter.offset.w1"), d, param("inter.offset.b1"), L.zfeat, d, nullptr, n_in,
                      d, d, EPI_RELU});
            }
            {
                StageTimer t(h, 2, s);
                launch_combine_center(c.model, g, sin, W, L.logits, L.zfeat, L.zmean, rels, rel_c, n_rel, d,
                                      L.states, L.dflag, s);
            }
            if (q2b) {
                {
                    StageTimer t(h, 1, s);
                    gemm({L.zmean, d, param("inter.offset.w2"), d, param("inter.offset.b2"), L.gate, d, nullptr,
                          st.count, d, d, EPI_NONE});
                }
                StageTimer t(h, 2, s);
                launch_combine_offset(g, sin, W, L.gate, rels, h->rel_o_sp, n_rel, d, L.states, L.dflag, s);
            }
        }
    }

    const int tq = score_row_pad(c.model);
    const int n_rows_pad = ((p.n_score_rows + tq - 1) / tq) * tq;
    const int d_score = logice ? 2 * d : d;    // LogicE scores its 2d bound coordinates as one vector
    {
        StageTimer t(h, 3, s);
        launch_pack(c.model, P + p.off_score_src, mlp ? P + p.off_score_neg : nullptr, p.n_score_rows, n_rows_pad,
                    L.states, W, d_score, L.qpack, L.cq, s);
    }
    float* dst = out_scores ? out_scores : L.scores;
    bool keyed = false;   // the scorer wrote chunk keys for top-k
    {
        StageTimer t(h, 4, s);
        ScoreArgs a{c.model, L.qpack, h->ent_blk, L.cq, h->ent_const, P + p.off_out_dest, p.n_score_rows,
                    p.n_quad_rows, p.n_pair_rows, d_score, N, h->n_blocks, c.gamma, c.center_reg, dst, N};
        a.dist_scale = logice ? 1.0f / (float)(2 * d) : cone ? h->cone_modulus : 1.0f;
        if (betae && h->dense_path != KGQ_DENSE_FP32) a.ent_planes = h->ent_planes;
        a.split_always = h->dense_path == KGQ_DENSE_BF16X3;
        a.part = L.score_ws;
        a.part_elems = L.score_ws_elems;
        if (out_idx) {
            a.chunk_key = L.chunk_key;
            a.key_ld = (N + kKeyChunk - 1) / kKeyChunk;
        }
        keyed = launch_score(a, s);
    }
    if (out_idx) {
        StageTimer t(h, 5, s);
        TopkArgs ta{};
        ta.scores = dst;
        ta.ld = N;
        ta.N = N;
        ta.n_rows = p.B;
        ta.k = k;
        ta.out_idx = out_idx;
        ta.out_score = out_score;
        for (int i = 0; i < 2; ++i) {
            ta.cand_idx[i] = L.cand_idx[i];
            ta.cand_score[i] = L.cand_score[i];
        }
        if (keyed) {
            ta.chunk_key = L.chunk_key;
            ta.key_ld = (N + kKeyChunk - 1) / kKeyChunk;
        }
        if (!launch_topk(ta, s)) return fail(h, KGQ_E_DEVICE, "top-k scratch buffers missing");
    }
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(h, KGQ_E_DEVICE, std::string("kernel launch: ") + hipGetErrorString(e));
    if (h->checked) {
        HIP_TRY(h, hipMemcpyAsync(L.hflag, L.dflag, sizeof(int), hipMemcpyDeviceToHost, s));
        HIP_TRY(h, hipStreamSynchronize(s));
        if (*L.hflag & kErrPadding)
            return fail(h, KGQ_E_INVALID_ARG, "a mixed-batch unused anchor/relation slot is not -1");
        if (*L.hflag & kErrRange) return fail(h, KGQ_E_OUT_OF_RANGE, "an anchor or relation id is out of range");
    }
    return KGQ_OK;
}

// Address of the static scratch array on the handle's device (current at
// the call): looked up once per device and kept for the process.
kgq_status noalloc_scratch_address(kgq_handle* h)
{
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    auto it = g_scratch_addr.find(h->cfg.device);
    if (it == g_scratch_addr.end()) {
        void* p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return fail(h, KGQ_E_DEVICE, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
        it = g_scratch_addr.emplace(h->cfg.device, static_cast<unsigned char*>(p)).first;
    }
    h->noalloc_scratch = it->second;
    return KGQ_OK;
}

// Lays the device buffers one lowered plan needs out in a region of `cap`
// bytes at `base` (256-byte aligned pieces), in the roles a lane's buffers
// play: plan image, error flag, state rows, dense-layer rows, intersection
// groups, packed queries, the score matrix when the caller does not supply
// one, and the top-k candidates of long rows. The scorers' chunk keys for top-k
// (which then reads only the chunks that can hold its answers), then the
// split-K and split-d workspaces of small batches get what is left, up to a
// lane's caps (the splitting code takes fewer slices when a workspace is
// smaller). Returns the
// bytes the required pieces need; *fits tells whether they fit `cap`.
int64_t carve_scratch(const kgq_handle* h, const Plan& p, int32_t k, bool need_scores, bool need_topk,
                      unsigned char* base, int64_t cap, Lane& V, int32_t** plan_dev, bool* fits)
{
    const kgq_config& c = h->cfg;
    const int64_t d = c.dim, N = c.n_entities, B = p.B;
    const int64_t W = (c.model == KGQ_GQE) ? d : 2 * d;
    int64_t off = 0;
    // (with base == nullptr only the sizes are wanted: the addresses formed
    // here are then never used)
    auto take = [&](int64_t bytes) -> unsigned char* {
        off = (off + 255) / 256 * 256;
        unsigned char* q = reinterpret_cast<unsigned char*>(reinterpret_cast<uintptr_t>(base) + (uintptr_t)off);
        off += std::max<int64_t>(bytes, 16);
        return q;
    };
    *plan_dev = reinterpret_cast<int32_t*>(take((int64_t)p.image.size() * 4));
    V.dflag = reinterpret_cast<int*>(take(sizeof(int)));
    V.states = reinterpret_cast<float*>(take((int64_t)p.n_state_rows * W * 4));
    const int64_t m = std::max(p.max_level, p.max_and_in), groups = p.max_and_groups;
    if (mlp_model(c.model)) {
        V.xbuf = reinterpret_cast<float*>(take(m * (c.model == KGQ_LOGICE ? 3 : 2) * d * 4));
        V.h1 = reinterpret_cast<float*>(take(m * 4 * d * 4));
        V.h2 = reinterpret_cast<float*>(take(m * 4 * d * 4));
        if (c.model == KGQ_CONE) {
            V.zmean = reinterpret_cast<float*>(take(groups * d * 4));
            V.gate = reinterpret_cast<float*>(take(groups * d * 4));
        }
    } else {
        V.h1 = reinterpret_cast<float*>(take(m * d * 4));
        if (c.model == KGQ_Q2B) {
            V.zfeat = reinterpret_cast<float*>(take(m * d * 4));
            V.zmean = reinterpret_cast<float*>(take(groups * d * 4));
            V.gate = reinterpret_cast<float*>(take(groups * d * 4));
        }
    }
    V.logits = reinterpret_cast<float*>(take(m * d * 4));
    const int tq = score_row_pad(c.model);
    const int64_t srows = ((int64_t)(p.n_score_rows + tq - 1) / tq) * tq;
    V.qpack = reinterpret_cast<float*>(take(srows * qpack_row_floats(c.model, (int)d) * 4));
    V.cq = reinterpret_cast<double*>(take(srows * 8));
    V.scores = need_scores ? reinterpret_cast<float*>(take(B * N * 4)) : nullptr;
    const int64_t ncand = need_topk ? topk_scratch_elems(B, N, k) : 0;
    for (int i = 0; i < 2; ++i) {
        V.cand_idx[i] = ncand ? reinterpret_cast<int32_t*>(take(ncand * 4)) : nullptr;
        V.cand_score[i] = ncand ? reinterpret_cast<float*>(take(ncand * 4)) : nullptr;
    }
    const int64_t required = off;
    *fits = required <= cap;
    V.gemm_ws = nullptr;
    V.gemm_ws_elems = 0;
    V.score_ws = nullptr;
    V.score_ws_elems = 0;
    V.chunk_key = nullptr;
    if (*fits) {
        // the scorers' chunk keys for top-k first, when they fit whole
        const int64_t key_bytes = B * ((N + kKeyChunk - 1) / kKeyChunk) * 4;
        if (need_topk && (off + 255) / 256 * 256 + key_bytes <= cap)
            V.chunk_key = reinterpret_cast<uint32_t*>(take(key_bytes));
        // optional workspaces, each from half of what is left
        const int64_t n_max = mlp_model(c.model) ? 4 * d : d;
        int64_t left = (cap - (off + 255) / 256 * 256) / 2 / 4 / 64 * 64;
        int64_t want = std::min<int64_t>(16 * 3 * B * n_max, (int64_t)16 * 128 * 4096);
        if (std::min(want, left) >= 64) {
            V.gemm_ws_elems = std::min(want, left);
            V.gemm_ws = reinterpret_cast<float*>(take(V.gemm_ws_elems * 4));
        }
        if (c.model != KGQ_BETAE) {
            const int64_t n_pad = h->n_blocks * kEntBlock;
            left = (cap - (off + 255) / 256 * 256) / 4 / 64 * 64;
            want = std::min<int64_t>(16 * 2 * (2 * B + 64) * n_pad, (int64_t)8 << 20);
            if (std::min(want, left) >= 64) {
                V.score_ws_elems = std::min(want, left);
                V.score_ws = reinterpret_cast<float*>(take(V.score_ws_elems * 4));
            }
        }
    }
    return required;
}

}  // namespace

// ===========================================================================
// Exported API
// ===========================================================================

extern "C" {

const char* kgq_status_string(kgq_status s)
{
    switch (s) {
    case KGQ_OK: return "ok";
    case KGQ_E_INVALID_ARG: return "invalid argument";
    case KGQ_E_OUT_OF_RANGE: return "id out of range";
    case KGQ_E_NOT_LOADED: return "parameters not loaded";
    case KGQ_E_UNSUPPORTED: return "unsupported structure for this model";
    case KGQ_E_NO_DEVICE: return "no device";
    case KGQ_E_OOM: return "out of memory";
    case KGQ_E_DEVICE: return "device error";
    }
    return "unknown status";
}

const char* kgq_last_error(const kgq_handle* h) { return h ? h->err.c_str() : ""; }

const char* kgq_create_error(void) { return g_create_error.c_str(); }

kgq_status kgq_structure_arity(int32_t structure_id, int32_t* n_anchors, int32_t* n_relations)
{
    const Program* g = builtin_program(KGQ_BETAE, structure_id);   // every built-in compiles for BetaE
    if (!g || !n_anchors || !n_relations) return KGQ_E_INVALID_ARG;
    *n_anchors = g->n_anchors;
    *n_relations = g->n_relations;
    return KGQ_OK;
}

kgq_status kgq_parse_structure(const char* text, kgq_node* nodes, int32_t capacity, int32_t* n_nodes)
{
    if (!text || !nodes || !n_nodes || capacity < 1) return KGQ_E_INVALID_ARG;
    std::vector<kgq_node> v;
    std::string err;
    if (!parse_graph(text, v, err) || (int32_t)v.size() > capacity) return KGQ_E_INVALID_ARG;
    std::memcpy(nodes, v.data(), v.size() * sizeof(kgq_node));
    *n_nodes = (int32_t)v.size();
    return KGQ_OK;
}

kgq_status kgq_compile_structure(kgq_handle* h, const kgq_node* nodes, int32_t n_nodes, int32_t* structure_id)
{
    if (!h) return KGQ_E_INVALID_ARG;
    if (!nodes || !structure_id) return fail(h, KGQ_E_INVALID_ARG, "nodes and structure_id must not be NULL");
    if ((int)h->compiled.size() >= KGQ_MAX_COMPILED)
        return fail(h, KGQ_E_INVALID_ARG, "the handle already holds KGQ_MAX_COMPILED compiled structures");
    std::unique_ptr<Program> g(new Program());
    std::string err;
    int st = 0;
    const int id = kNumStructures + (int)h->compiled.size();
    if (!compile_graph(h->cfg.model, nodes, n_nodes, "#" + std::to_string(id), *g, err, st))
        return fail(h, (kgq_status)st, err);
    if (max_batch_for(h, *g) < 1)
        return fail(h, KGQ_E_INVALID_ARG, "structure #" + std::to_string(id) +
                                              " needs more scratch for one query than the handle holds");
    h->table.push_back(g.get());
    h->compiled.push_back(std::move(g));
    *structure_id = id;
    return KGQ_OK;
}

kgq_status kgq_structure_info(const kgq_handle* h, int32_t structure_id, int32_t* info)
{
    if (!h || !info) return KGQ_E_INVALID_ARG;
    const Program* g = program_of(h, structure_id);
    if (!g) return KGQ_E_INVALID_ARG;
    if (!g->supported) return KGQ_E_UNSUPPORTED;
    info[0] = g->n_anchors;
    info[1] = g->n_relations;
    info[2] = g->n_terms;
    info[3] = (int32_t)g->ops.size();
    info[4] = g->and_stages;
    info[5] = program_launches(h->cfg.model, *g, true);
    info[6] = (int32_t)max_batch_for(h, *g);
    info[7] = g->negation ? 1 : 0;
    return KGQ_OK;
}

kgq_status kgq_create(const kgq_config* cfg, kgq_handle** out)
{
    g_create_error.clear();
    auto bad = [](const std::string& m) {
        g_create_error = m;
        return KGQ_E_INVALID_ARG;
    };
    if (!cfg || !out) return bad("cfg and out must not be NULL");
    *out = nullptr;
    const kgq_config& c = *cfg;
    if (c.model < KGQ_GQE || c.model > KGQ_LOGICE) return bad("unknown model " + std::to_string(c.model));
    if (c.model == KGQ_LOGICE && (c.tnorm < KGQ_TNORM_PRODUCT || c.tnorm > KGQ_TNORM_LUKASIEWICZ))
        return bad("unknown t-norm " + std::to_string(c.tnorm));
    if (c.model == KGQ_CONE && c.entity_dtype != KGQ_F32) return bad("ConE takes a float32 entity table");
    if (c.model == KGQ_CONE && !(c.center_reg >= 0.f && c.center_reg <= 1.f)) return bad("center_reg outside [0, 1]");
    if (c.dim < 4 || c.dim > 4096 || c.dim % 4) return bad("dim must be a multiple of 4 in [4, 4096]");
    if (c.n_entities < 1 || c.n_entities > 0x7fffffffLL) return bad("n_entities outside [1, 2^31-1]");
    if (c.n_relations < 1) return bad("n_relations must be >= 1");
    if (c.entity_dtype != KGQ_F32 && c.entity_dtype != KGQ_BF16) return bad("unknown entity_dtype");
    if (c.max_batch < 1 || c.max_batch > (1 << 20)) return bad("max_batch outside [1, 2^20]");
    if (!(c.gamma == c.gamma)) return bad("gamma is NaN");
    if (c.model == KGQ_Q2B && !(c.center_reg >= 0.f && c.center_reg <= 1.f)) return bad("center_reg outside [0, 1]");
    if (c.device < -1) return bad("device must be >= -1");
    if (c.concurrency < 0 || c.concurrency > 64) return bad("concurrency outside [0, 64]");

    std::unique_ptr<kgq_handle> h(new kgq_handle());
    h->cfg = c;
    h->dry = c.device < 0;
    const char* env = std::getenv("KGQ_CHECKED");
    h->checked = env && env[0] == '1';
    build_specs(h.get());
    build_table(h.get());
    if (h->dry) {
        *out = h.release();
        return KGQ_OK;
    }
    int n_dev = 0;
    if (hipGetDeviceCount(&n_dev) != hipSuccess || n_dev <= c.device) {
        g_create_error = "no HIP device " + std::to_string(c.device);
        return KGQ_E_NO_DEVICE;
    }
    if (hipSetDevice(c.device) != hipSuccess) {
        g_create_error = "hipSetDevice failed";
        return KGQ_E_NO_DEVICE;
    }
    kgq_status s = allocate_all(h.get());
    if (s == KGQ_OK) s = noalloc_scratch_address(h.get());
    if (s != KGQ_OK) {
        g_create_error = h->err;
        free_all(h.get());
        return s;
    }
    *out = h.release();
    return KGQ_OK;
}

kgq_status kgq_rank_answers(kgq_handle* h, int32_t batch, const float* scores, int64_t ld,
                            const int32_t* ans_offsets, const int32_t* ans_ids, const int32_t* ans_hard,
                            int32_t* out_rank, double* out_metrics, void* stream)
{
    static_assert(KGQ_MAX_ANSWERS == kMaxAnswers, "answer-list limit");
    if (!h) return KGQ_E_INVALID_ARG;
    if (!scores || !ans_offsets || !ans_ids || !out_rank)
        return fail(h, KGQ_E_INVALID_ARG, "scores, ans_offsets, ans_ids and out_rank must not be NULL");
    if (batch < 1) return fail(h, KGQ_E_INVALID_ARG, "batch must be >= 1");
    const int64_t N = h->cfg.n_entities;
    if (ld < N) return fail(h, KGQ_E_INVALID_ARG, "ld must be >= n_entities");
    if (h->dry) return fail(h, KGQ_E_NO_DEVICE, "validation-only handle (device = -1)");
    HIP_TRY(h, hipSetDevice(h->cfg.device));
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    Lane* L = nullptr;
    kgq_status st = acquire_lane(h, s, &L);
    if (st != KGQ_OK) return st;
    if (h->checked) launch_clear_flag(L->dflag, s);
    launch_rank_answers(scores, ld, N, batch, ans_offsets, ans_ids, ans_hard, out_rank, out_metrics, L->dflag, s);
    HIP_TRY(h, hipGetLastError());
    L->done_live = hipEventRecord(L->done, s) == hipSuccess;
    if (h->checked) {
        HIP_TRY(h, hipMemcpyAsync(L->hflag, L->dflag, sizeof(int), hipMemcpyDeviceToHost, s));
        HIP_TRY(h, hipStreamSynchronize(s));
        if (*L->hflag & kErrAnswers)
            return fail(h, KGQ_E_INVALID_ARG, "an answer list is longer than KGQ_MAX_ANSWERS or of negative length");
        if (*L->hflag & kErrRange) return fail(h, KGQ_E_OUT_OF_RANGE, "an answer id is out of range");
    }
    return KGQ_OK;
}

kgq_status kgq_memory(const kgq_handle* h, int64_t* param_bytes, int64_t* scratch_bytes)
{
    if (!h) return KGQ_E_INVALID_ARG;
    if (param_bytes) *param_bytes = h->bytes_params;
    if (scratch_bytes) *scratch_bytes = h->bytes_total - h->bytes_params;
    return KGQ_OK;
}

kgq_status kgq_destroy(kgq_handle* h)
{
    if (!h) return KGQ_OK;
    free_all(h);
    delete h;
    return KGQ_OK;
}

kgq_status kgq_execute_mixed_noalloc(kgq_handle* h, int32_t batch, const int32_t* structure_ids,
                                     const int32_t* anchors, const int32_t* relations, int32_t k, float* out_scores,
                                     int32_t* out_topk_idx, float* out_topk_score, void* stream)
{
    static_assert(KGQ_NOALLOC_SCRATCH_BYTES % 256 == 0, "scratch size");
    if (!h) return KGQ_E_INVALID_ARG;
    if (!structure_ids) return fail(h, KGQ_E_INVALID_ARG, "structure_ids must not be NULL");
    kgq_status st = check_outputs(h, batch, anchors, relations, k, out_scores, out_topk_idx, out_topk_score);
    if (st != KGQ_OK) return st;
    std::string err;
    int es = 0;
    Plan plan;
    if (!lower(h->cfg.model, batch, structure_ids, 0, 3, 3, true, h->table, plan, err, es))
        return fail(h, (kgq_status)es, err);
    st = check_capacity(h, plan);   // the plan is staged through a lane's pinned slots
    if (st != KGQ_OK) return st;
    // every device buffer of the call lives in the static array: size check
    // first (no address needed for it, so a validation-only handle checks it too)
    Lane V;
    int32_t* plan_dev = nullptr;
    bool fits = false;
    const int64_t need = carve_scratch(h, plan, k, out_scores == nullptr, out_topk_idx != nullptr, nullptr,
                                       KGQ_NOALLOC_SCRATCH_BYTES, V, &plan_dev, &fits);
    if (!fits)
        return fail(h, KGQ_E_INVALID_ARG,
                    "the batch needs " + std::to_string(need) + " bytes of device scratch, more than the " +
                        std::to_string((int64_t)KGQ_NOALLOC_SCRATCH_BYTES) +
                        " of the static array (KGQ_NOALLOC_SCRATCH_BYTES); split it" +
                        (out_scores ? std::string() : std::string(" or pass out_scores")));
    if (h->dry) return fail(h, KGQ_E_NO_DEVICE, "validation-only handle (device = -1)");
    if (!h->noalloc_scratch) return fail(h, KGQ_E_DEVICE, "no static scratch address for this device");
    HIP_TRY(h, hipSetDevice(h->cfg.device));
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    carve_scratch(h, plan, k, out_scores == nullptr, out_topk_idx != nullptr, h->noalloc_scratch,
                  KGQ_NOALLOC_SCRATCH_BYTES, V, &plan_dev, &fits);
    // The lane provides the pinned plan staging, the host flag and the
    // ordering against the lane's previous call; its device buffers are not
    // used.
    Lane* L = nullptr;
    st = acquire_lane(h, s, &L);
    if (st != KGQ_OK) return st;
    V.hflag = L->hflag;
    // the array keeps the last call's contents: the error flag must start at zero
    launch_clear_flag(V.dflag, s);
    const int slot = kNumStructures + L->ring_next;
    L->ring_next ^= 1;
    st = upload_plan(h, *L, plan, slot, s, plan_dev);
    if (st != KGQ_OK) return st;
    st = run_plan(h, V, plan, plan_dev, anchors, relations, 3, 3, 0, 0, true, k, out_scores, out_topk_idx,
                  out_topk_score, s);
    L->slot_event_live[slot] = hipEventRecord(L->slot_event[slot], s) == hipSuccess;
    L->done_live = hipEventRecord(L->done, s) == hipSuccess;
    return st;
}

kgq_status kgq_set_checked(kgq_handle* h, int32_t on)
{
    if (!h) return KGQ_E_INVALID_ARG;
    h->checked = on != 0;
    return KGQ_OK;
}

// BetaE first-layer tables (see proj1_ent / proj1_rel): rebuilt whenever
// one of their inputs is (re)loaded and all of them are present.
static const char* entity_param_name(int model)
{
    switch (model) {
    case KGQ_BETAE: return "entity.alpha_beta";
    case KGQ_CONE: return "entity.axis";
    case KGQ_LOGICE: return "entity.bounds";
    default: return "entity";
    }
}

// First-layer tables of the projection MLP (BetaE, ConE, LogicE): the layer
// is linear in its input, so W1 x + b1 for an anchor entity's state splits
// into an entity table and a relation table. BetaE and ConE add the relation
// to the state (x = state + Rel[r]: both tables use all of W1); LogicE
// concatenates it (x = [state; Rel[r]]: the entity table uses W1's first 2d
// columns, the relation table the last d).
static kgq_status build_proj1(kgq_handle* h)
{
    const kgq_config& c = h->cfg;
    h->proj1_ready = false;
    for (const char* n : {entity_param_name(c.model), "relation", "proj.w1", "proj.b1"})
        if (!h->loaded[n]) return KGQ_OK;
    const int d = c.dim;
    const bool logice = c.model == KGQ_LOGICE;
    const int in_w = logice ? 3 * d : 2 * d;
    const float* w1 = h->dparam.at("proj.w1");
    launch_gemm({h->ent_rm, 2 * d, w1, in_w, nullptr, h->proj1_ent, 4 * d, nullptr, (int)c.n_entities, 4 * d, 2 * d,
                 EPI_NONE}, nullptr);
    if (logice)
        launch_gemm({h->dparam.at("relation"), d, w1 + 2 * d, in_w, h->dparam.at("proj.b1"), h->proj1_rel, 4 * d,
                     nullptr, c.n_relations, 4 * d, d, EPI_NONE}, nullptr);
    else
        launch_gemm({h->dparam.at("relation"), 2 * d, w1, 2 * d, h->dparam.at("proj.b1"), h->proj1_rel, 4 * d,
                     nullptr, c.n_relations, 4 * d, 2 * d, EPI_NONE}, nullptr);
    HIP_TRY(h, hipGetLastError());
    HIP_TRY(h, hipStreamSynchronize(nullptr));
    h->proj1_ready = true;
    return KGQ_OK;
}

kgq_status kgq_load_params(kgq_handle* h, const char* name, const void* src, size_t nbytes, int32_t dtype,
                           int32_t src_is_device)
{
    if (!h) return KGQ_E_INVALID_ARG;
    if (!name) return fail(h, KGQ_E_INVALID_ARG, "name must not be NULL");
    auto it = h->specs.find(name);
    if (it == h->specs.end()) return fail(h, KGQ_E_INVALID_ARG, std::string("unknown parameter '") + name + "'");
    const ParamSpec& ps = it->second;
    const int want_dtype = ps.entity ? h->cfg.entity_dtype : KGQ_F32;
    if (dtype != want_dtype)
        return fail(h, KGQ_E_INVALID_ARG, std::string("parameter '") + name + "' expects dtype " +
                                              (want_dtype == KGQ_BF16 ? "bf16" : "f32"));
    const size_t elem = dtype == KGQ_BF16 ? 2 : 4;
    const size_t want = (size_t)(ps.rows * ps.cols) * elem;
    if (nbytes != want)
        return fail(h, KGQ_E_INVALID_ARG, std::string("parameter '") + name + "' needs " + std::to_string(want) +
                                              " bytes, got " + std::to_string(nbytes));
    if (!src) return fail(h, KGQ_E_INVALID_ARG, "src must not be NULL");
    if (h->dry) {
        h->loaded[name] = true;
        return KGQ_OK;
    }
    HIP_TRY(h, hipSetDevice(h->cfg.device));
    const hipMemcpyKind kind = src_is_device ? hipMemcpyDeviceToDevice : hipMemcpyHostToDevice;
    const kgq_config& c = h->cfg;
    if (!ps.entity) {
        float* dst = h->dparam.at(name);
        HIP_TRY(h, hipMemcpy(dst, src, nbytes, kind));
        if (c.model == KGQ_Q2B && std::strcmp(name, "relation.offset_raw") == 0) {
            launch_softplus(dst, h->rel_o_sp, ps.rows * ps.cols, nullptr);
            HIP_TRY(h, hipGetLastError());
            HIP_TRY(h, hipStreamSynchronize(nullptr));
        }
        auto split = [&](const float* w, int64_t rows, int64_t cols) -> kgq_status {
            auto pl = h->wplanes.find(w);
            if (pl == h->wplanes.end()) return KGQ_OK;
            launch_split_planes(w, pl->second, rows, cols, nullptr);
            HIP_TRY(h, hipGetLastError());
            HIP_TRY(h, hipStreamSynchronize(nullptr));
            return KGQ_OK;
        };
        kgq_status st = split(dst, ps.rows, ps.cols);
        if (st != KGQ_OK) return st;
        if (c.model == KGQ_CONE) {
            // the two set functions' first layers, stacked for one GEMM
            const size_t half_w = (size_t)2 * c.dim * c.dim, half_b = (size_t)c.dim;
            if (!std::strcmp(name, "inter.axis.w1")) HIP_TRY(h, hipMemcpy(h->int_cat_w, dst, nbytes, hipMemcpyDeviceToDevice));
            if (!std::strcmp(name, "inter.arg.w1"))
                HIP_TRY(h, hipMemcpy(h->int_cat_w + half_w, dst, nbytes, hipMemcpyDeviceToDevice));
            if (!std::strcmp(name, "inter.axis.w1") || !std::strcmp(name, "inter.arg.w1"))
                if ((st = split(h->int_cat_w, 2 * (int64_t)c.dim, 2 * (int64_t)c.dim)) != KGQ_OK) return st;
            if (!std::strcmp(name, "inter.axis.b1")) HIP_TRY(h, hipMemcpy(h->int_cat_b, dst, nbytes, hipMemcpyDeviceToDevice));
            if (!std::strcmp(name, "inter.arg.b1"))
                HIP_TRY(h, hipMemcpy(h->int_cat_b + half_b, dst, nbytes, hipMemcpyDeviceToDevice));
            if (!std::strcmp(name, "modulus")) HIP_TRY(h, hipMemcpy(&h->cone_modulus, dst, sizeof(float), hipMemcpyDeviceToHost));
        }
        h->loaded[name] = true;
        if (mlp_model(c.model) && (!std::strcmp(name, "relation") || !std::strcmp(name, "proj.w1") ||
                                   !std::strcmp(name, "proj.b1")))
            return build_proj1(h);
        return KGQ_OK;
    }
    // entity table: stage, then build the derived layouts
    void* stage = nullptr;
    hipError_t e = hipMalloc(&stage, nbytes);
    if (e != hipSuccess) return fail(h, KGQ_E_OOM, "staging buffer for the entity table");
    e = hipMemcpy(stage, src, nbytes, kind);
    if (e == hipSuccess) {
        const int bf16 = dtype == KGQ_BF16;
        if (c.model == KGQ_BETAE) {
            launch_betae_entity_prep(stage, bf16, c.n_entities, c.dim, h->n_blocks, h->ent_rm, h->ent_blk,
                                     h->ent_const, nullptr);
            if (h->ent_planes)
                launch_split_planes(h->ent_blk, h->ent_planes, h->n_blocks * kEntBlock, 2 * (int64_t)c.dim, nullptr);
        }
        else if (c.model == KGQ_CONE)
            launch_cone_entity_prep(static_cast<const float*>(stage), c.n_entities, c.dim, h->n_blocks, h->ent_rm,
                                    h->ent_blk, nullptr);
        else
            launch_relayout_points(stage, bf16, c.n_entities, c.model == KGQ_LOGICE ? 2 * c.dim : c.dim,
                                   h->n_blocks, h->ent_rm, h->ent_blk, nullptr);
        e = hipGetLastError();
        if (e == hipSuccess) e = hipStreamSynchronize(nullptr);
    }
    (void)hipFree(stage);
    if (e != hipSuccess) return fail(h, KGQ_E_DEVICE, std::string("entity table load: ") + hipGetErrorString(e));
    h->loaded[name] = true;
    if (mlp_model(c.model)) return build_proj1(h);
    return KGQ_OK;
}

kgq_status kgq_execute(kgq_handle* h, int32_t structure_id, int32_t batch, const int32_t* anchors,
                       const int32_t* relations, int32_t k, float* out_scores, int32_t* out_topk_idx,
                       float* out_topk_score, void* stream)
{
    if (!h) return KGQ_E_INVALID_ARG;
    const Program* g = program_of(h, structure_id);
    if (!g) return fail(h, KGQ_E_INVALID_ARG, "unknown structure id " + std::to_string(structure_id));
    if (!g->supported)
        return fail(h, KGQ_E_UNSUPPORTED, "structure " + g->name + " needs negation (BetaE only)");
    kgq_status st = check_outputs(h, batch, anchors, relations, k, out_scores, out_topk_idx, out_topk_score);
    if (st != KGQ_OK) return st;
    // built-in structures keep their lowered plan per batch size in a slot
    // of their own; compiled ones are lowered into the ring slots
    const bool cached = structure_id < kNumStructures;
    std::unique_ptr<Plan> fresh;
    if (!cached || h->dry) {
        fresh.reset(new Plan());
        std::string err;
        int es = 0;
        if (!lower(h->cfg.model, batch, nullptr, structure_id, g->n_anchors, g->n_relations, false, h->table, *fresh,
                   err, es))
            return fail(h, (kgq_status)es, err);
        st = check_capacity(h, *fresh);
        if (st != KGQ_OK) return st;
    }
    if (h->dry) return fail(h, KGQ_E_NO_DEVICE, "validation-only handle (device = -1)");
    HIP_TRY(h, hipSetDevice(h->cfg.device));
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    Lane* L = nullptr;
    st = acquire_lane(h, s, &L);
    if (st != KGQ_OK) return st;
    const Plan* plan = nullptr;
    int slot;
    if (cached) {
        slot = structure_id;
        if (L->cached_B[slot] != batch || !L->cached_plan[slot]) {
            std::unique_ptr<Plan> p(new Plan());
            std::string err;
            int es = 0;
            if (!lower(h->cfg.model, batch, nullptr, structure_id, g->n_anchors, g->n_relations, false, h->table, *p,
                       err, es))
                return fail(h, (kgq_status)es, err);
            st = check_capacity(h, *p);
            if (st != KGQ_OK) return st;
            st = upload_plan(h, *L, *p, slot, s);
            if (st != KGQ_OK) return st;
            L->cached_plan[slot] = std::move(p);
            L->cached_B[slot] = batch;
        }
        plan = L->cached_plan[slot].get();
    } else {
        slot = kNumStructures + L->ring_next;
        L->ring_next ^= 1;
        st = upload_plan(h, *L, *fresh, slot, s);
        if (st != KGQ_OK) return st;
        plan = fresh.get();
    }
    const int32_t* P = L->plan_dev + (int64_t)slot * h->plan_words;
    st = run_plan(h, *L, *plan, P, anchors, relations, g->n_anchors, g->n_relations, g->n_anchors, g->n_relations,
                  false, k, out_scores, out_topk_idx, out_topk_score, s);
    L->slot_event_live[slot] = hipEventRecord(L->slot_event[slot], s) == hipSuccess;
    L->done_live = hipEventRecord(L->done, s) == hipSuccess;
    return st;
}

kgq_status kgq_execute_mixed(kgq_handle* h, int32_t batch, const int32_t* structure_ids, const int32_t* anchors,
                             const int32_t* relations, int32_t k, float* out_scores, int32_t* out_topk_idx,
                             float* out_topk_score, void* stream)
{
    if (!h) return KGQ_E_INVALID_ARG;
    if (!structure_ids) return fail(h, KGQ_E_INVALID_ARG, "structure_ids must not be NULL");
    kgq_status st = check_outputs(h, batch, anchors, relations, k, out_scores, out_topk_idx, out_topk_score);
    if (st != KGQ_OK) return st;
    std::string err;
    int es = 0;
    Plan plan;
    if (!lower(h->cfg.model, batch, structure_ids, 0, 3, 3, true, h->table, plan, err, es))
        return fail(h, (kgq_status)es, err);
    st = check_capacity(h, plan);
    if (st != KGQ_OK) return st;
    if (h->dry) return fail(h, KGQ_E_NO_DEVICE, "validation-only handle (device = -1)");
    HIP_TRY(h, hipSetDevice(h->cfg.device));
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    Lane* L = nullptr;
    st = acquire_lane(h, s, &L);
    if (st != KGQ_OK) return st;
    const int slot = kNumStructures + L->ring_next;
    L->ring_next ^= 1;
    st = upload_plan(h, *L, plan, slot, s);
    if (st != KGQ_OK) return st;
    const int32_t* P = L->plan_dev + (int64_t)slot * h->plan_words;
    st = run_plan(h, *L, plan, P, anchors, relations, 3, 3, 0, 0, true, k, out_scores, out_topk_idx,
                  out_topk_score, s);
    L->slot_event_live[slot] = hipEventRecord(L->slot_event[slot], s) == hipSuccess;
    L->done_live = hipEventRecord(L->done, s) == hipSuccess;
    return st;
}

kgq_status kgq_describe_plan(const kgq_handle* h, int32_t batch, const int32_t* structure_ids, int32_t* counts)
{
    if (!h || !structure_ids || !counts || batch < 1) return KGQ_E_INVALID_ARG;
    Plan p;
    std::string err;
    int es = 0;
    if (!lower(h->cfg.model, batch, structure_ids, 0, kMaxSlots, kMaxSlots, true, h->table, p, err, es)) {
        const_cast<kgq_handle*>(h)->err = err;
        return (kgq_status)es;
    }
    counts[0] = p.n_anchor_chains;
    counts[1] = p.n_groups;
    counts[2] = p.n_int_in;
    for (int l = 0; l < 4; ++l) counts[3 + l] = p.level_rows[l];
    counts[7] = p.n_score_rows;
    counts[8] = p.n_pair_rows / 2;
    counts[9] = plan_launches(p, true);
    counts[10] = p.n_and_stages;
    counts[11] = p.n_quad_rows / 4;
    counts[12] = p.n_state_rows;
    return KGQ_OK;
}

kgq_status kgq_dense(kgq_handle* h, const float* x, int32_t M, int32_t K, const float* w, const float* b, int32_t N,
                     int32_t act, float* y, void* stream)
{
    if (!h) return KGQ_E_INVALID_ARG;
    if (!x || !w || !y) return fail(h, KGQ_E_INVALID_ARG, "x, w and y must not be NULL");
    if (M < 1 || N < 1 || K < 4 || K % 4) return fail(h, KGQ_E_INVALID_ARG, "need M, N >= 1 and K a multiple of 4");
    if (act < EPI_NONE || act > EPI_BETA_REG) return fail(h, KGQ_E_INVALID_ARG, "unknown activation");
    if ((reinterpret_cast<uintptr_t>(x) | reinterpret_cast<uintptr_t>(w)) & 15)
        return fail(h, KGQ_E_INVALID_ARG, "x and w must be 16-byte aligned");
    if (h->dry) return fail(h, KGQ_E_NO_DEVICE, "validation-only handle (device = -1)");
    HIP_TRY(h, hipSetDevice(h->cfg.device));
    hipStream_t s = reinterpret_cast<hipStream_t>(stream);
    GemmArgs g{x, K, w, K, b, y, N, nullptr, M, N, K, act};
    // the bf16 matrix-core path needs w's planes: split into a
    // stream-ordered buffer that lives until the layer has run
    uint16_t* planes = nullptr;
    g.bf16x3_always = h->dense_path == KGQ_DENSE_BF16X3;
    if (h->dense_path != KGQ_DENSE_FP32 && gemm_shape_takes_bf16x3(M, N, K, K, g.bf16x3_always)) {
        HIP_TRY(h, hipMallocAsync((void**)&planes, (size_t)3 * N * plane_ld(K) * sizeof(uint16_t), s));
        launch_split_planes(w, planes, N, K, s);
        g.Wp = planes;
    }
    {
        StageTimer t(h, 1, s);
        launch_gemm(g, s);
    }
    if (planes) HIP_TRY(h, hipFreeAsync(planes, s));
    HIP_TRY(h, hipGetLastError());
    return KGQ_OK;
}

kgq_status kgq_set_dense_path(kgq_handle* h, int32_t path)
{
    if (!h) return KGQ_E_INVALID_ARG;
    if (path < KGQ_DENSE_AUTO || path > KGQ_DENSE_BF16X3) return fail(h, KGQ_E_INVALID_ARG, "unknown dense path");
    h->dense_path = path;
    return KGQ_OK;
}

kgq_status kgq_profile_enable(kgq_handle* h, int32_t on)
{
    if (!h) return KGQ_E_INVALID_ARG;
    if (h->dry) return fail(h, KGQ_E_NO_DEVICE, "validation-only handle (device = -1)");
    if (on && !h->prof_ref) {
        // time origin for kgq_profile_intervals, on the null stream
        HIP_TRY(h, hipEventCreate(&h->prof_ref));
        HIP_TRY(h, hipEventRecord(h->prof_ref, nullptr));
    }
    if (on < 0 || on >= (1 << KGQ_NUM_STAGES)) return fail(h, KGQ_E_INVALID_ARG, "stage mask out of range");
    if (!on && h->prof) prof_collect(h);
    h->prof = on;
    return KGQ_OK;
}

kgq_status kgq_profile_read(kgq_handle* h, int32_t stage, double* total_ms, int64_t* launches)
{
    if (!h || stage < 0 || stage >= KGQ_NUM_STAGES || !total_ms || !launches) return KGQ_E_INVALID_ARG;
    if (h->dry) return fail(h, KGQ_E_NO_DEVICE, "validation-only handle (device = -1)");
    prof_collect(h);
    *total_ms = h->prof_ms[stage];
    *launches = h->prof_n[stage];
    return KGQ_OK;
}

kgq_status kgq_profile_reset(kgq_handle* h)
{
    if (!h) return KGQ_E_INVALID_ARG;
    if (h->dry) return KGQ_OK;
    prof_collect(h);
    for (int i = 0; i < KGQ_NUM_STAGES; ++i) {
        h->prof_ms[i] = 0.0;
        h->prof_n[i] = 0;
        h->prof_iv[i].clear();
    }
    return KGQ_OK;
}

kgq_status kgq_profile_intervals(kgq_handle* h, int32_t stage, double* out, int64_t cap, int64_t* n)
{
    if (!h || stage < 0 || stage >= KGQ_NUM_STAGES || !n || (cap > 0 && !out)) return KGQ_E_INVALID_ARG;
    if (h->dry) return fail(h, KGQ_E_NO_DEVICE, "validation-only handle (device = -1)");
    prof_collect(h);
    const std::vector<double>& v = h->prof_iv[stage];
    *n = (int64_t)v.size() / 2;
    const int64_t m = *n < cap ? *n : cap;
    for (int64_t i = 0; i < 2 * m; ++i) out[i] = v[(size_t)i];
    return KGQ_OK;
}

}  // extern "C"
