// pactshard.hip -- host side of libpactshard: argument validation, the
// per-step scalars, the segment batching and the launches.  The C ABI and
// its contract are in include/pactshard.h.
#include "pactshard.h"

#include <algorithm>
#include <cmath>
#include <cstring>
#include <mutex>

#include "launch.h"

// What the kernels and the batching below rely on.
static_assert(pact::kBlock % 64 == 0 && pact::kBlock <= 1024, "whole waves of 64, one block");
static_assert(pact::kVec == 4, "the binary32 vector path moves 16-byte vectors of four elements");
static_assert(pact::kTile % (pact::kBlock * 8) == 0,
              "a BF16-state tile is whole rows of 16-byte vectors of eight elements");
static_assert((pact::kLanes & (pact::kLanes - 1)) == 0, "lane = workgroup & (kLanes - 1)");
static_assert(pact::kLaneStride * sizeof(uint64_t) >= 128, "lanes sit in separate cache lines");
static_assert((uint64_t)pact::kTile * 4 <= (1ull << 31), "a tile's byte offsets fit the 32-bit buffer offset");
static_assert(pact::kSegsPerLaunch >= 1, "a launch takes at least one segment");

namespace {

thread_local int g_last_hip_error = 0;

constexpr uint64_t kIndexLimit = 1ull << 56;  // indices must stay below the tag bits
constexpr uint32_t kMaxSegments = 1u << 24;     // keeps every slot and lane index in 32 bits

int fail_hip(hipError_t e) {
    g_last_hip_error = static_cast<int>(e);
    return PACT_EHIP;
}

// ---------------------------------------------------------------------------
// One view over either kind of shard: the five array slots are param, grad,
// exp_avg, exp_avg_sq and the bf16 working copy; a BF16 shard has 2-byte
// elements and no working copy.
// ---------------------------------------------------------------------------
enum Slot { kP = 0, kG = 1, kM = 2, kV = 3, kB = 4, kSlots = 5 };

struct View {
    const void* arr[kSlots];
    uint32_t esize[kSlots];  // bytes per element (0: the shard has no such array)
    uint64_t numel;
    uint64_t goff;
    const pact_segment* segs;
    uint32_t num_segs;
    uint32_t num_hypers;
    const pact_hyper* hypers;
    uint64_t* digest;
    void* workspace;
    uint64_t workspace_bytes;
    void* stream;
};

template <typename S>
View common_view(const S* s) {
    View v;
    v.arr[kP] = s->param;
    v.arr[kG] = s->grad;
    v.arr[kM] = s->exp_avg;
    v.arr[kV] = s->exp_avg_sq;
    v.numel = s->numel;
    v.goff = s->global_offset;
    v.segs = s->segs;
    v.num_segs = s->num_segs;
    v.num_hypers = s->num_hypers;
    v.hypers = s->hypers;
    v.digest = s->digest_dev;
    v.workspace = s->workspace;
    v.workspace_bytes = s->workspace_bytes;
    v.stream = s->stream;
    return v;
}

View view_of(const pact_shard* s) {
    View v = common_view(s);
    v.arr[kB] = s->param_bf16;
    v.esize[kP] = v.esize[kG] = v.esize[kM] = v.esize[kV] = 4;
    v.esize[kB] = 2;
    return v;
}

View view_of(const pact_shard_bf16* s) {
    View v = common_view(s);
    v.arr[kB] = nullptr;
    v.esize[kP] = v.esize[kG] = v.esize[kM] = v.esize[kV] = 2;
    v.esize[kB] = 0;
    return v;
}

// ---------------------------------------------------------------------------
// validation
// ---------------------------------------------------------------------------
bool finite(float x) { return std::isfinite(x); }

bool hyper_ok(const pact_hyper& h) {
    return finite(h.lr) && finite(h.beta1) && finite(h.beta2) && finite(h.eps) && finite(h.weight_decay) &&
           h.lr >= 0.0f && h.beta1 >= 0.0f && h.beta1 < 1.0f && h.beta2 >= 0.0f && h.beta2 < 1.0f &&
           h.eps > 0.0f && h.weight_decay >= 0.0f;
}

bool aligned(const void* p, uintptr_t a) { return (reinterpret_cast<uintptr_t>(p) & (a - 1)) == 0; }

struct Span {
    uintptr_t lo, hi;  // [lo, hi)
};

// The buffers of one call: the five arrays, the result slots, the workspace.
constexpr int kMaxSpans = kSlots + 2;

bool overlaps(const Span* spans, int n) {
    for (int i = 0; i < n; ++i) {
        for (int j = i + 1; j < n; ++j) {
            if (spans[i].lo < spans[j].hi && spans[j].lo < spans[i].hi) return true;
        }
    }
    return false;
}

// Result slots that accumulate partial sums (one per segment, or one), and
// the workspace bytes their lanes take.
uint64_t result_slots(const View& s) { return s.segs ? (uint64_t)s.num_segs : 1; }

uint64_t workspace_need(const View& s) {
    return result_slots(s) * pact::kLanes * pact::kLaneStride * sizeof(uint64_t);
}

// Which array slots a mode touches.
struct Uses {
    bool slot[kSlots];
};

// Checks the shard for a mode; `out` is the digest destination.  Returns 0 or
// a PACT_E* code.  Reads no device memory and makes no HIP call.
int validate(const View& s, const Uses& use, const uint64_t* out, uint64_t* nslots) {
    if (out == nullptr) return PACT_EINVAL;
    const uint64_t n = s.numel;
    for (int k = 0; k < kSlots; ++k) {
        if (use.slot[k] && s.esize[k] == 0) return PACT_EINVAL;  // this shard kind has no such array
        if (use.slot[k] && n > 0 && s.arr[k] == nullptr) return PACT_EINVAL;
    }
    if (s.goff >= kIndexLimit || n > kIndexLimit - s.goff) return PACT_ERANGE;
    if (n > (UINT64_MAX / 4)) return PACT_ERANGE;
    uint64_t tiles = (n + pact::kTile - 1) / pact::kTile;
    if (s.segs != nullptr) {
        if (s.num_segs == 0 || s.num_segs > kMaxSegments) return PACT_EINVAL;
        uint64_t prev_end = 0;
        tiles = 0;
        for (uint32_t k = 0; k < s.num_segs; ++k) {
            const pact_segment& sg = s.segs[k];
            if (sg.reserved != 0 || sg.offset < prev_end || sg.length > n || sg.offset > n - sg.length) {
                return PACT_EINVAL;
            }
            prev_end = sg.offset + sg.length;
            tiles += (sg.length + pact::kTile - 1) / pact::kTile;  // tiles never straddle segments
        }
    }
    // A dispatch counts its work-items in 32 bits, so one launch holds at most
    // UINT32_MAX / kBlock tiles; the total bounds every launch's share.
    if (tiles > (uint64_t)(UINT32_MAX / pact::kBlock)) return PACT_ERANGE;
    if (!aligned(out, 8)) return PACT_EALIGN;
    for (int k = 0; k < kSlots; ++k) {
        if (use.slot[k] && !aligned(s.arr[k], s.esize[k])) return PACT_EALIGN;
    }
    const uint64_t slots = s.segs ? (uint64_t)s.num_segs + 1 : 1;
    if (s.workspace != nullptr) {
        if (!aligned(s.workspace, 8)) return PACT_EALIGN;
        if (s.workspace_bytes < workspace_need(s)) return PACT_EINVAL;
    }
    Span spans[kMaxSpans];
    int nspans = 0;
    auto add = [&](const void* ptr, uint64_t bytes) {
        if (ptr && bytes) {
            const uintptr_t lo = reinterpret_cast<uintptr_t>(ptr);
            spans[nspans++] = {lo, lo + bytes};
        }
    };
    for (int k = 0; k < kSlots; ++k) {
        if (use.slot[k]) add(s.arr[k], n * s.esize[k]);
    }
    add(out, slots * 8);
    if (s.workspace != nullptr) add(s.workspace, workspace_need(s));
    for (int k = 0; k < nspans; ++k) {
        if (spans[k].hi < spans[k].lo) return PACT_ERANGE;  // wraps the address space
    }
    if (overlaps(spans, nspans)) return PACT_EOVERLAP;
    *nslots = slots;
    return PACT_OK;
}

// ---------------------------------------------------------------------------
// per-step scalars: beta^t by t double multiplications from 1, the derived
// values in double, one binary32 rounding each
// ---------------------------------------------------------------------------

// beta^t as the plain loop computes it: pow <- pow * beta, t times, stopping
// once a product equals its predecessor (every later product then equals it
// too, so the value is the one t multiplications give; only 1 - beta^t is
// used, so the sign of a zero power does not matter).  A training run calls
// with t, t+1, t+2, ...: each thread remembers the last power it reached for
// a few betas and carries on from there, so a call costs O(1)
// multiplications instead of O(t) (about 10^5 per segment at step 10^5).
double beta_power(double beta, uint64_t t) {
    struct Memo {
        uint64_t beta_bits;
        uint64_t t;      // multiplications done
        double pow;
        bool fixed;      // the product has stopped changing
        bool used;
    };
    constexpr int kMemo = 8;
    thread_local Memo memo[kMemo] = {};
    thread_local int victim = 0;
    uint64_t bits;
    std::memcpy(&bits, &beta, sizeof bits);
    Memo* m = nullptr;
    for (Memo& e : memo) {
        if (e.used && e.beta_bits == bits && e.t <= t) {
            m = &e;
            break;
        }
    }
    if (m == nullptr) {
        m = &memo[victim];
        victim = (victim + 1) % kMemo;
        *m = Memo{bits, 0, 1.0, false, true};
    }
    if (m->fixed) return m->pow;
    double pow = m->pow;
    uint64_t k = m->t;
    bool fixed = false;
    for (; k < t; ++k) {
        const double next = pow * beta;
        fixed = next == pow;
        pow = next;
        if (fixed) {
            ++k;
            break;
        }
    }
    // keep the furthest point reached (a call for an earlier step restarts)
    if (k >= m->t) {
        m->t = k;
        m->pow = pow;
        m->fixed = fixed;
    }
    return pow;
}

pact::StepScalars step_scalars(const pact_hyper& h, uint64_t t) {
    const double beta1 = h.beta1, beta2 = h.beta2;
    const double pow1 = beta_power(beta1, t);
    const double pow2 = beta_power(beta2, t);
    const double lr = h.lr, wd = h.weight_decay;
    pact::StepScalars sc;
    sc.beta1 = h.beta1;
    sc.beta2 = h.beta2;
    sc.eps = h.eps;
    sc.decay = static_cast<float>(1.0 - lr * wd);
    sc.omb1 = static_cast<float>(1.0 - beta1);
    sc.omb2 = static_cast<float>(1.0 - beta2);
    sc.step_size = static_cast<float>(lr / (1.0 - pow1));
    sc.rs_bc2 = static_cast<float>(1.0 / std::sqrt(1.0 - pow2));
    return sc;
}

// ---------------------------------------------------------------------------
// enqueue one mode over the shard's segments
// ---------------------------------------------------------------------------
struct SegWork {
    uint64_t first, count;
    pact::StepScalars sc;
};

// The shard's segments as units of work, formed one at a time (a call keeps
// no table of its own): the whole shard without a segment table, else one
// per table entry.  `single` and `step` give the scalars when need_hyper.
struct SegSource {
    const View* s;
    const pact_hyper* single;
    uint64_t step;
    bool need_hyper;

    size_t count() const { return s->segs ? (size_t)s->num_segs : (s->numel > 0 ? 1 : 0); }
    SegWork at(size_t k) const {
        SegWork w{0, s->numel, {}};
        const pact_hyper* h = single;
        if (s->segs) {
            const pact_segment& sg = s->segs[k];
            w.first = sg.offset;
            w.count = sg.length;  // empty segments keep their slot (digest 0)
            h = &s->hypers[sg.hyper_index];
        }
        if (need_hyper) w.sc = step_scalars(*h, step);
        return w;
    }
};

// Every segment's hyperparameter index and set, when the mode needs them;
// PACT_EINVAL before anything is enqueued if one is bad.
int check_segment_hypers(const View& s) {
    if (s.segs == nullptr) return PACT_OK;
    if (s.hypers == nullptr) return PACT_EINVAL;
    for (uint32_t k = 0; k < s.num_segs; ++k) {
        const uint32_t hi = s.segs[k].hyper_index;
        if (hi >= s.num_hypers || !hyper_ok(s.hypers[hi])) return PACT_EINVAL;
    }
    return PACT_OK;
}

bool is_bf16_state(pact::Mode m) { return m == pact::Mode::CommitBf16State || m == pact::Mode::DigestBf16State; }

// Whether a segment starting at element `first` can take the vector path:
// 16-byte aligned in every array the mode moves as 16-byte vectors, 8-byte in
// the bf16 working copy.
bool vector_ok(pact::Mode mode, const View& s, uint64_t first) {
    auto at = [&](int k, uintptr_t a) {
        return aligned(static_cast<const char*>(s.arr[k]) + first * s.esize[k], a);
    };
    switch (mode) {
        case pact::Mode::Bf16Digest:
            return at(kB, 8);
        case pact::Mode::GradGuard:
            return at(kG, 16);
        case pact::Mode::StateDigest:
        case pact::Mode::DigestBf16State:
            return at(kP, 16) && at(kM, 16) && at(kV, 16);
        case pact::Mode::CommitBf16State:
            return at(kP, 16) && at(kG, 16) && at(kM, 16) && at(kV, 16);
        case pact::Mode::Commit:
        case pact::Mode::CommitZeroGrad:
            return at(kP, 16) && at(kG, 16) && at(kM, 16) && at(kV, 16) && at(kB, 8);
    }
    return false;
}

// workspace_clean: the caller vouches that the workspace lanes are zero (the
// finish kernel leaves them so), and the clearing launch is skipped.
int run(pact::Mode mode, const View& s, const SegSource& work, uint64_t* out, uint64_t nslots,
        bool workspace_clean = false) {
    hipStream_t stream = static_cast<hipStream_t>(s.stream);
    uint64_t* lanes = static_cast<uint64_t*>(s.workspace);
    const uint32_t nres = (uint32_t)result_slots(s);
    hipError_t e = hipSuccess;
    if (!(workspace_clean && lanes != nullptr)) {
        e = pact::launch_clear(out, lanes, nres, (uint32_t)nslots, stream);
        if (e != hipSuccess) return fail_hip(e);
    }

    pact::Arrays a;
    pact::ArraysBf16 ab;
    std::memset(&a, 0, sizeof a);
    std::memset(&ab, 0, sizeof ab);
    if (is_bf16_state(mode)) {
        ab.p = static_cast<uint16_t*>(const_cast<void*>(s.arr[kP]));
        ab.g = static_cast<const uint16_t*>(s.arr[kG]);
        ab.m = static_cast<uint16_t*>(const_cast<void*>(s.arr[kM]));
        ab.v = static_cast<uint16_t*>(const_cast<void*>(s.arr[kV]));
        ab.goff = s.goff;
        ab.digest = out;
        ab.lanes = lanes;
    } else {
        a.p = static_cast<float*>(const_cast<void*>(s.arr[kP]));
        a.g = static_cast<const float*>(s.arr[kG]);
        a.g_zero = const_cast<float*>(a.g);  // written only by Mode::CommitZeroGrad
        a.m = static_cast<float*>(const_cast<void*>(s.arr[kM]));
        a.v = static_cast<float*>(const_cast<void*>(s.arr[kV]));
        a.b = static_cast<uint16_t*>(const_cast<void*>(s.arr[kB]));
        a.goff = s.goff;
        a.digest = out;
        a.lanes = lanes;
    }

    const bool per_segment = s.segs != nullptr;
    const size_t nwork = work.count();
    for (size_t first = 0; first < nwork; first += pact::kSegsPerLaunch) {
        const size_t cnt = std::min<size_t>(pact::kSegsPerLaunch, nwork - first);
        pact::Batch b;
        std::memset(&b, 0, sizeof b);
        b.nseg = (uint32_t)cnt;
        b.slot0 = (uint32_t)first;
        b.per_segment = per_segment ? 1u : 0u;
        uint64_t tiles = 0;
        for (size_t k = 0; k < cnt; ++k) {
            const SegWork w = work.at(first + k);
            b.tile_begin[k] = tiles;
            tiles += (w.count + pact::kTile - 1) / pact::kTile;
            b.elem_begin[k] = w.first;
            b.elem_count[k] = w.count;
            b.sc[k] = w.sc;
            b.vec_ok[k] = vector_ok(mode, s, w.first) ? 1u : 0u;
        }
        b.tile_begin[cnt] = tiles;
        if (tiles == 0) continue;
        e = is_bf16_state(mode) ? pact::launch_batch_bf16(mode, ab, b, (uint32_t)tiles, stream)
                                : pact::launch_batch(mode, a, b, (uint32_t)tiles, stream);
        if (e != hipSuccess) return fail_hip(e);
    }
    if (lanes != nullptr || per_segment) {
        e = pact::launch_finish(out, lanes, nres, per_segment, stream);
        if (e != hipSuccess) return fail_hip(e);
    }
    return PACT_OK;
}

// ---------------------------------------------------------------------------
// Static scratch of pact_adamw_commit_static: the digest lanes of up to
// PACT_STATIC_MAX_SEGMENTS result slots in device memory the library holds
// for the life of the process, one copy per GPU.  In host code `scratch`
// names a host-side stand-in, not a device address: the device address of
// each GPU's copy is looked up once per device and only that is used.
// ---------------------------------------------------------------------------
constexpr uint64_t kStaticScratchWords = (uint64_t)PACT_STATIC_MAX_SEGMENTS * pact::kLanes * pact::kLaneStride;
constexpr uint64_t kStaticScratchBytes = kStaticScratchWords * sizeof(uint64_t);
constexpr int kMaxDevices = 64;

std::mutex g_scratch_mu;
void* g_scratch_dev[kMaxDevices] = {};

}  // namespace

static __device__ __align__(256) uint64_t scratch[kStaticScratchWords];

namespace {

// The device address of the GPU's copy of `scratch` for the device `stream`
// belongs to (the current device for the null stream), looked up with that
// device current on the first call for it.
int static_scratch_ptr(void* stream, void** out) {
    int dev = -1;
    hipError_t e = stream ? hipStreamGetDevice(static_cast<hipStream_t>(stream), &dev) : hipGetDevice(&dev);
    if (e != hipSuccess) return fail_hip(e);
    if (dev < 0 || dev >= kMaxDevices) return PACT_EINVAL;
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (g_scratch_dev[dev] == nullptr) {
        int cur = -1;
        e = hipGetDevice(&cur);
        if (e != hipSuccess) return fail_hip(e);
        if (cur != dev && (e = hipSetDevice(dev)) != hipSuccess) return fail_hip(e);
        void* ptr = nullptr;
        e = hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch));
        if (cur != dev) {
            const hipError_t back = hipSetDevice(cur);
            if (e == hipSuccess) e = back;
        }
        if (e != hipSuccess) return fail_hip(e);
        if (ptr == nullptr) return fail_hip(hipErrorInvalidSymbol);
        g_scratch_dev[dev] = ptr;
    }
    *out = g_scratch_dev[dev];
    return PACT_OK;
}

// A commit mode: check step and hyperparameters, validate, enqueue.  With
// static_scratch the digest lanes are the library's static array (the
// caller's workspace must be absent).
int commit(pact::Mode mode, View s, uint64_t step, const pact_hyper* hyper, const Uses& use,
           bool workspace_clean = false, bool static_scratch = false) {
    if (step == 0) return PACT_EINVAL;
    if (s.segs == nullptr && (hyper == nullptr || !hyper_ok(*hyper))) return PACT_EINVAL;
    uint64_t nslots = 0;
    int rc = validate(s, use, s.digest, &nslots);
    if (rc != PACT_OK) return rc;
    rc = check_segment_hypers(s);
    if (rc != PACT_OK) return rc;
    if (static_scratch) {
        if (s.workspace != nullptr) return PACT_EINVAL;
        if (result_slots(s) > PACT_STATIC_MAX_SEGMENTS) return PACT_ESCRATCH;
        void* lanes = nullptr;
        rc = static_scratch_ptr(s.stream, &lanes);
        if (rc != PACT_OK) return rc;
        s.workspace = lanes;
        s.workspace_bytes = kStaticScratchBytes;
        workspace_clean = false;  // shared by every call on the GPU: always cleared first
    }
    const SegSource work{&s, hyper, step, true};
    return run(mode, s, work, s.digest, nslots, workspace_clean);
}

// A mode that only reads the shard: validate, enqueue.
int measure(pact::Mode mode, const View& s, const Uses& use, uint64_t* out) {
    uint64_t nslots = 0;
    int rc = validate(s, use, out, &nslots);
    if (rc != PACT_OK) return rc;
    const SegSource work{&s, nullptr, 0, false};
    return run(mode, s, work, out, nslots);
}

}  // namespace

extern "C" {

int64_t pact_digest_slots(const pact_shard* s) {
    if (s == nullptr) return PACT_EINVAL;
    return s->segs ? (int64_t)s->num_segs + 1 : 1;
}

int64_t pact_workspace_bytes(const pact_shard* s) {
    if (s == nullptr) return PACT_EINVAL;
    return (int64_t)workspace_need(view_of(s));
}

int64_t pact_digest_slots_bf16(const pact_shard_bf16* s) {
    if (s == nullptr) return PACT_EINVAL;
    return s->segs ? (int64_t)s->num_segs + 1 : 1;
}

int64_t pact_workspace_bytes_bf16(const pact_shard_bf16* s) {
    if (s == nullptr) return PACT_EINVAL;
    return (int64_t)workspace_need(view_of(s));
}

int pact_adamw_commit_ex(const pact_shard* s, uint64_t step, const pact_hyper* hyper, uint32_t flags) {
    if (s == nullptr || (flags & ~(PACT_COMMIT_ZERO_GRAD | PACT_COMMIT_WORKSPACE_CLEAN)) != 0) return PACT_EINVAL;
    const Uses use = {{true, true, true, true, true}};
    const pact::Mode mode = (flags & PACT_COMMIT_ZERO_GRAD) ? pact::Mode::CommitZeroGrad : pact::Mode::Commit;
    return commit(mode, view_of(s), step, hyper, use, (flags & PACT_COMMIT_WORKSPACE_CLEAN) != 0);
}

int pact_adamw_commit(const pact_shard* s, uint64_t step, const pact_hyper* hyper) {
    return pact_adamw_commit_ex(s, step, hyper, 0u);
}

int pact_adamw_commit_static(const pact_shard* s, uint64_t step, const pact_hyper* hyper, uint32_t flags) {
    if (s == nullptr || (flags & ~PACT_COMMIT_ZERO_GRAD) != 0) return PACT_EINVAL;
    const Uses use = {{true, true, true, true, true}};
    const pact::Mode mode = (flags & PACT_COMMIT_ZERO_GRAD) ? pact::Mode::CommitZeroGrad : pact::Mode::Commit;
    return commit(mode, view_of(s), step, hyper, use, false, true);
}

int pact_grad_guard(const pact_shard* s, uint64_t* dev_out) {
    if (s == nullptr) return PACT_EINVAL;
    const Uses use = {{false, true, false, false, false}};
    return measure(pact::Mode::GradGuard, view_of(s), use, dev_out);
}

int pact_shard_digest(const pact_shard* s) {
    if (s == nullptr) return PACT_EINVAL;
    const Uses use = {{true, false, true, true, false}};
    return measure(pact::Mode::StateDigest, view_of(s), use, s->digest_dev);
}

int pact_bf16_digest(const pact_shard* s, uint64_t* dev_out) {
    if (s == nullptr) return PACT_EINVAL;
    const Uses use = {{false, false, false, false, true}};
    return measure(pact::Mode::Bf16Digest, view_of(s), use, dev_out);
}

int pact_adamw_commit_bf16(const pact_shard_bf16* s, uint64_t step, const pact_hyper* hyper) {
    if (s == nullptr) return PACT_EINVAL;
    const Uses use = {{true, true, true, true, false}};
    return commit(pact::Mode::CommitBf16State, view_of(s), step, hyper, use);
}

int pact_shard_digest_bf16(const pact_shard_bf16* s) {
    if (s == nullptr) return PACT_EINVAL;
    const Uses use = {{true, false, true, true, false}};
    return measure(pact::Mode::DigestBf16State, view_of(s), use, s->digest_dev);
}

int pact_arena_plan(uint64_t numel, uint64_t spacing, pact_arena_layout* out) {
    if (out == nullptr) return PACT_EINVAL;
    constexpr uint64_t kAlign = 2ull << 20;
    // every size below stays far from 2^64: numel < 2^56 keeps 4 * numel < 2^58
    if (numel >= kIndexLimit || spacing > (1ull << 58)) return PACT_ERANGE;
    auto round_up = [](uint64_t x) { return (x + kAlign - 1) / kAlign * kAlign; };
    const uint64_t f32 = round_up(numel * 4), b16 = round_up(numel * 2);
    uint64_t sp = spacing;
    if (sp == 0) sp = (4 * f32 + b16 > PACT_ARENA_PACK_BELOW) ? PACT_ARENA_SPACING : f32;
    sp = round_up(std::max(sp, f32));
    out->spacing = sp;
    for (int k = 0; k < 5; ++k) out->offset[k] = (uint64_t)k * sp;
    out->pool_bytes = 4 * sp + b16;
    return PACT_OK;
}

int pact_stream_probe_grid(const float* in0, const float* in1, const float* in2, const float* in3, float* out0,
                           float* out2, float* out3, uint16_t* out_half, uint64_t n, uint32_t workgroups,
                           void* stream) {
    if (n == 0) return PACT_OK;
    if (!in0 || !in1 || !in2 || !in3 || !out0 || !out2 || !out3 || !out_half || (n % pact::kVec) != 0) {
        return PACT_EINVAL;
    }
    if (!aligned(in0, 16) || !aligned(in1, 16) || !aligned(in2, 16) || !aligned(in3, 16) || !aligned(out0, 16) ||
        !aligned(out2, 16) || !aligned(out3, 16) || !aligned(out_half, 8)) {
        return PACT_EALIGN;
    }
    const uint64_t tiles = (n + pact::kTile - 1) / pact::kTile;
    if (tiles > (uint64_t)(UINT32_MAX / pact::kBlock) || workgroups > UINT32_MAX / pact::kBlock) return PACT_ERANGE;
    hipError_t e = pact::launch_probe(in0, in1, in2, in3, out0, out2, out3, out_half, n, workgroups,
                                      static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return fail_hip(e);
    return PACT_OK;
}

int pact_stream_probe(const float* in0, const float* in1, const float* in2, const float* in3, float* out0,
                      float* out2, float* out3, uint16_t* out_half, uint64_t n, void* stream) {
    return pact_stream_probe_grid(in0, in1, in2, in3, out0, out2, out3, out_half, n, 0u, stream);
}

const char* pact_strerror(int code) {
    switch (code) {
        case PACT_OK: return "ok";
        case PACT_EINVAL: return "invalid argument";
        case PACT_EALIGN: return "misaligned pointer";
        case PACT_EOVERLAP: return "buffers overlap";
        case PACT_ERANGE: return "index range reaches the digest tag bits (2^56), wraps, or exceeds one launch grid";
        case PACT_EHIP: return "HIP call failed";
        case PACT_ESCRATCH: return "more segments than the library's static scratch holds";
        default: return "unknown error";
    }
}

int pact_last_hip_error(void) { return g_last_hip_error; }

int pact_version(void) { return 300; }

}  // extern "C"
