// Host side of the C ABI declared in include/conduit.h: argument validation,
// buffer layout in HBM, host-known ring state, sticky device error flags, and
// kernel launches on the caller's stream.
#include <cstdio>
#include <cstring>
#include <mutex>
#include <string>

#include "common.h"
#include "gae_plan.h"

using namespace conduit;

namespace {

thread_local std::string g_last_error;

conduit_status fail(conduit_status s, const std::string& msg) {
    g_last_error = msg;
    return s;
}

}  // namespace

// the error reporting of the other host sources (common.h)
conduit_status conduit::report_error(conduit_status s, const char* msg) { return fail(s, msg); }

namespace {

conduit_status hip_fail(hipError_t e, const char* what) {
    return fail(CONDUIT_EDEVICE, std::string(what) + ": " + hipGetErrorString(e));
}

// ---------------------------------------------------------------------------
// Sticky error words.  One page of pinned, device-visible host memory holds
// kErrKinds words per slot; slot 0 serves the stand-alone calls.  Kernels store
// a 1 into the word of the error kind they hit.  The page is never freed (a
// kernel still in flight may write it), so it lives for the process.
// ---------------------------------------------------------------------------
constexpr int kErrSlots = 512;
std::mutex g_err_mu;
uint32_t* g_err_host = nullptr;  // host view
uint32_t* g_err_dev = nullptr;   // device view of the same page
bool g_slot_used[kErrSlots];

conduit_status err_page() {
    if (g_err_host) return CONDUIT_OK;
    void* p = nullptr;
    hipError_t e = hipHostMalloc(&p, sizeof(uint32_t) * kErrKinds * kErrSlots, hipHostMallocMapped);
    if (e != hipSuccess) return hip_fail(e, "hipHostMalloc(error flags)");
    void* d = nullptr;
    e = hipHostGetDevicePointer(&d, p, 0);
    if (e != hipSuccess) return hip_fail(e, "hipHostGetDevicePointer(error flags)");
    std::memset(p, 0, sizeof(uint32_t) * kErrKinds * kErrSlots);
    g_err_host = static_cast<uint32_t*>(p);
    g_err_dev = static_cast<uint32_t*>(d);
    g_slot_used[0] = true;
    return CONDUIT_OK;
}

conduit_status err_slot_acquire(int* slot) {
    std::lock_guard<std::mutex> lk(g_err_mu);
    conduit_status s = err_page();
    if (s != CONDUIT_OK) return s;
    for (int i = 1; i < kErrSlots; ++i) {
        if (!g_slot_used[i]) {
            g_slot_used[i] = true;
            std::memset(g_err_host + i * kErrKinds, 0, sizeof(uint32_t) * kErrKinds);
            *slot = i;
            return CONDUIT_OK;
        }
    }
    return fail(CONDUIT_ENOMEM, "too many live buffers (error-flag slots exhausted)");
}

void err_slot_release(int slot) {
    std::lock_guard<std::mutex> lk(g_err_mu);
    if (slot > 0 && slot < kErrSlots) g_slot_used[slot] = false;
}

const char* kErrText[kErrKinds] = {
    "priority update index outside [0, size)",
    "gather index outside [0, size)",
    "sample from a tree whose total priority is 0",
    "sequence length outside [0, max_len]",
    "permutation entry outside [0, n_src)",
    "GAE segment never published by its workgroup (GAE calls overlapping on one GPU?)",
    "sum-tree descent found no child",
    "ragged ingest offsets decreasing or outside [0, src_elems]",
};

// Returns ESTATE if any flag of `slot` is set (no synchronisation).
conduit_status check_flags(int slot) {
    if (!g_err_host) return CONDUIT_OK;
    volatile uint32_t* w = g_err_host + slot * kErrKinds;
    std::string msg;
    for (int k = 0; k < kErrKinds; ++k) {
        if (w[k]) {
            if (!msg.empty()) msg += "; ";
            msg += kErrText[k];
        }
    }
    if (msg.empty()) return CONDUIT_OK;
    return fail(CONDUIT_ESTATE, "device-side error flagged earlier: " + msg);
}

uint32_t* err_words(int slot) { return g_err_dev + slot * kErrKinds; }

// Stand-alone calls: make sure the flag page exists, then report slot 0.
conduit_status standalone_flags() {
    {
        std::lock_guard<std::mutex> lk(g_err_mu);
        conduit_status st = err_page();
        if (st != CONDUIT_OK) return st;
    }
    return check_flags(0);
}

struct DeviceGuard {
    int prev = -1;
    explicit DeviceGuard(int dev) {
        if (hipGetDevice(&prev) != hipSuccess) prev = -1;
        if (prev != dev) (void)hipSetDevice(dev);
    }
    ~DeviceGuard() {
        int cur = -1;
        if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
    }
};

constexpr size_t kAlign = 256;

size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

int64_t round64(int64_t x) { return (x + 63) / 64 * 64; }

int dtype_size(conduit_dtype d) {
    switch (d) {
        case CONDUIT_U8: return 1;
        case CONDUIT_I32: return 4;
        case CONDUIT_F32: return 4;
        case CONDUIT_BF16: return 2;
    }
    return 0;
}

// Everything create() needs, derived from the parameters.
struct Layout {
    int64_t row_bytes = 0, max_len = 0;
    int depth = 0;
    int64_t nodes[kMaxLevels + 1] = {};
    size_t off_state = 0, off_obs = 0, off_aux = 0, off_action = 0, off_reward = 0, off_done = 0;
    size_t off_episode = 0, off_step = 0, off_length = 0, off_leaves = 0, off_level[kMaxLevels + 1] = {};
    size_t total = 0;
    // payload in pinned host memory: observation then auxiliary column
    bool host_payload = false;
    size_t host_obs = 0, host_aux = 0;
};

conduit_status make_layout(int64_t capacity, const int64_t* shape, int32_t ndim, conduit_dtype dt,
                           const conduit_buffer_opts& o, Layout* L) {
    if (capacity < 1 || capacity > 0x7fffffffLL) return fail(CONDUIT_EINVAL, "capacity must be in [1, 2^31-1]");
    if (!shape || ndim < 1 || ndim > 8) return fail(CONDUIT_EINVAL, "obs_shape must have 1..8 dimensions");
    const int es = dtype_size(dt);
    if (es == 0) return fail(CONDUIT_EINVAL, "unknown obs dtype");
    int64_t elems = 1;
    for (int i = 0; i < ndim; ++i) {
        if (shape[i] < 1 || shape[i] > (1LL << 31)) return fail(CONDUIT_EINVAL, "obs_shape entries must be positive");
        elems *= shape[i];
        if (elems > (1LL << 34)) return fail(CONDUIT_EINVAL, "observation too large");
    }
    L->row_bytes = elems * es;
    if (L->row_bytes % 4 != 0) return fail(CONDUIT_EINVAL, "observation size must be a multiple of 4 bytes");
    if (o.alpha_den < 1 || o.alpha_den > 8 || o.alpha_num < 0 || o.alpha_num > o.alpha_den)
        return fail(CONDUIT_EINVAL, "alpha must be alpha_num/alpha_den with 0 <= num <= den <= 8");
    if (!(o.beta >= 0.0) || o.beta > 1e6) return fail(CONDUIT_EINVAL, "beta must be a finite value >= 0");
    if (o.frame_stack < 1 || o.frame_stack > 16) return fail(CONDUIT_EINVAL, "frame_stack must be in [1, 16]");
    if (o.frame_stack > capacity) return fail(CONDUIT_EINVAL, "frame_stack larger than capacity");
    if (o.action_bytes < 0 || o.action_bytes > 256) return fail(CONDUIT_EINVAL, "action_bytes must be in [0, 256]");
    if (o.prioritized != 0 && o.prioritized != 1) return fail(CONDUIT_EINVAL, "prioritized must be 0 or 1");
    if (o.ragged) {
        if (ndim != 1 || es != 4) return fail(CONDUIT_EINVAL, "ragged buffers need obs_shape {max_len} of a 4-byte type");
        if (shape[0] % 4 != 0) return fail(CONDUIT_EINVAL, "ragged max_len must be a multiple of 4");
        if (o.aux_elem_bytes != 0 && o.aux_elem_bytes != 4) return fail(CONDUIT_EINVAL, "aux_elem_bytes must be 0 or 4");
        if (o.frame_stack != 1) return fail(CONDUIT_EINVAL, "ragged buffers do not stack frames");
        L->max_len = shape[0];
    } else if (o.aux_elem_bytes != 0) {
        return fail(CONDUIT_EINVAL, "aux_elem_bytes needs a ragged buffer");
    }
    if (o.payload_placement == CONDUIT_PLACE_HOST_PAGEABLE)
        return fail(CONDUIT_EINVAL, "kernels cannot address pageable memory: place the payload in HBM or pinned host memory");
    if (o.payload_placement != CONDUIT_PLACE_HBM && o.payload_placement != CONDUIT_PLACE_HOST_PINNED)
        return fail(CONDUIT_EINVAL, "unknown payload placement");
    if (o.weight_norm != CONDUIT_WNORM_BATCH && o.weight_norm != CONDUIT_WNORM_BUFFER)
        return fail(CONDUIT_EINVAL, "weight_norm must be CONDUIT_WNORM_BATCH or CONDUIT_WNORM_BUFFER");
    if (o.single_stream != 0 && o.single_stream != 1) return fail(CONDUIT_EINVAL, "single_stream must be 0 or 1");
    // tree shape
    L->nodes[0] = capacity;
    int d = 0;
    do {
        ++d;
        L->nodes[d] = (L->nodes[d - 1] + kFanout - 1) / kFanout;
    } while (L->nodes[d] > 1);
    L->depth = d;
    // arena layout
    size_t off = 0;
    auto take = [&](size_t bytes) {
        size_t at = off;
        off += align_up(bytes);
        return at;
    };
    const size_t C = (size_t)capacity;
    const size_t obs_bytes = C * (size_t)L->row_bytes;
    const size_t aux_bytes = o.ragged && o.aux_elem_bytes ? C * (size_t)L->max_len * (size_t)o.aux_elem_bytes : 0;
    L->off_state = take(sizeof(DeviceState));
    L->host_payload = o.payload_placement == CONDUIT_PLACE_HOST_PINNED;
    if (L->host_payload) {
        L->host_obs = align_up(obs_bytes);
        L->host_aux = align_up(aux_bytes);
    } else {
        L->off_obs = take(obs_bytes);
        L->off_aux = aux_bytes ? take(aux_bytes) : 0;
    }
    L->off_action = o.action_bytes ? take(C * (size_t)o.action_bytes) : 0;
    L->off_reward = take(C * 4);
    L->off_done = take(C);
    L->off_episode = take(C * 4);
    L->off_step = take(C * 4);
    L->off_length = o.ragged ? take(C * 4) : 0;
    if (o.prioritized) {
        L->off_leaves = take((size_t)round64(capacity) * 4);
        for (int l = 1; l <= d; ++l) L->off_level[l] = take((size_t)round64(L->nodes[l]) * 8);
    }
    L->total = off;
    return CONDUIT_OK;
}

}  // namespace

struct conduit_buffer {
    int device = 0;
    int64_t capacity = 0;
    conduit_dtype obs_dtype = CONDUIT_U8;
    conduit_buffer_opts opts{};
    Layout layout;
    uint8_t* arena = nullptr;
    bool owns_arena = false;
    uint8_t* host_payload = nullptr;  // pinned host allocation of a host-placed payload
    uint8_t* obs = nullptr;
    uint8_t* aux = nullptr;
    uint8_t* action = nullptr;
    float* reward = nullptr;
    uint8_t* done = nullptr;
    uint32_t* episode = nullptr;
    int32_t* step = nullptr;
    int32_t* length = nullptr;
    DeviceState* state = nullptr;
    TreeView tree{};
    int err_slot = -1;
    int64_t head = 0, size = 0, total = 0;
};

BufferGeometry conduit::buffer_geometry(const conduit_buffer* b) {
    BufferGeometry g;
    g.row_bytes = b->layout.row_bytes;
    g.frame_stack = b->opts.frame_stack;
    g.action_bytes = b->opts.action_bytes;
    g.ragged = b->opts.ragged != 0;
    g.prioritized = b->opts.prioritized != 0;
    g.capacity = b->capacity;
    g.head = b->head;
    g.obs = b->obs;
    return g;
}

// Device (or mapped host) address and size in bytes of one column; a column
// the buffer does not hold has size 0.
static conduit_status column_span(const conduit_buffer* b, conduit_column col, int32_t level, uint8_t** base,
                                  int64_t* bytes) {
    const Layout& L = b->layout;
    const int64_t C = b->capacity;
    uint8_t* p = nullptr;
    int64_t n = 0;
    switch (col) {
        case CONDUIT_COL_OBS: p = b->obs; n = C * L.row_bytes; break;
        case CONDUIT_COL_ACTION: p = b->action; n = b->action ? C * b->opts.action_bytes : 0; break;
        case CONDUIT_COL_REWARD: p = reinterpret_cast<uint8_t*>(b->reward); n = C * 4; break;
        case CONDUIT_COL_DONE: p = b->done; n = C; break;
        case CONDUIT_COL_EPISODE: p = reinterpret_cast<uint8_t*>(b->episode); n = C * 4; break;
        case CONDUIT_COL_STEP: p = reinterpret_cast<uint8_t*>(b->step); n = C * 4; break;
        case CONDUIT_COL_LENGTH: p = reinterpret_cast<uint8_t*>(b->length); n = b->length ? C * 4 : 0; break;
        case CONDUIT_COL_AUX: p = b->aux; n = b->aux ? C * L.max_len * b->opts.aux_elem_bytes : 0; break;
        case CONDUIT_COL_LEAVES:
            p = reinterpret_cast<uint8_t*>(b->tree.leaves);
            n = b->opts.prioritized ? C * 4 : 0;
            break;
        case CONDUIT_COL_TREE:
            if (!b->opts.prioritized || level < 1 || level > L.depth) return fail(CONDUIT_EINVAL, "no such tree level");
            p = reinterpret_cast<uint8_t*>(b->tree.level[level]);
            n = L.nodes[level] * 8;
            break;
        case CONDUIT_COL_MAX_PRIO: p = reinterpret_cast<uint8_t*>(&b->state->max_prio); n = 4; break;
        default: return fail(CONDUIT_EINVAL, "unknown column");
    }
    *base = p;
    *bytes = p ? n : 0;
    return CONDUIT_OK;
}

// The checkpoint header of `b`: layout fields, ring state and the section
// table (sections in column order, each at a multiple of 256 bytes).
static_assert(sizeof(conduit_ckpt_section) == 24 && sizeof(conduit_ckpt_header) == 344,
              "checkpoint header layout is part of the image format");

static void ckpt_header(const conduit_buffer* b, conduit_ckpt_header* h) {
    std::memset(h, 0, sizeof(*h));
    std::memcpy(h->magic, CONDUIT_CKPT_MAGIC, sizeof(h->magic));
    h->version = CONDUIT_CKPT_VERSION;
    h->capacity = b->capacity;
    h->row_bytes = b->layout.row_bytes;
    h->max_len = b->layout.max_len;
    h->obs_dtype = (int32_t)b->obs_dtype;
    h->prioritized = b->opts.prioritized;
    h->alpha_num = b->opts.alpha_num;
    h->alpha_den = b->opts.alpha_den;
    h->action_bytes = b->opts.action_bytes;
    h->ragged = b->opts.ragged;
    h->aux_elem_bytes = b->opts.aux_elem_bytes;
    h->head = b->head;
    h->size = b->size;
    h->total = (uint64_t)b->total;
    static const conduit_column order[] = {CONDUIT_COL_OBS,     CONDUIT_COL_ACTION, CONDUIT_COL_REWARD,
                                           CONDUIT_COL_DONE,    CONDUIT_COL_EPISODE, CONDUIT_COL_STEP,
                                           CONDUIT_COL_LENGTH,  CONDUIT_COL_AUX,    CONDUIT_COL_LEAVES,
                                           CONDUIT_COL_MAX_PRIO};
    static_assert(sizeof(order) / sizeof(order[0]) == CONDUIT_CKPT_MAX_SECTIONS, "one section per stored column");
    size_t off = align_up(sizeof(*h));
    for (conduit_column c : order) {
        uint8_t* base = nullptr;
        int64_t n = 0;
        (void)column_span(b, c, 0, &base, &n);
        if (n == 0) continue;
        conduit_ckpt_section& sec = h->section[h->n_sections++];
        sec.column = (int32_t)c;
        sec.offset = (int64_t)off;
        sec.bytes = n;
        off = align_up(off + (size_t)n);
    }
    h->image_bytes = off;
}

extern "C" {

void conduit_buffer_opts_default(conduit_buffer_opts* o) {
    if (!o) return;
    o->prioritized = 1;
    o->alpha_num = 3;
    o->alpha_den = 5;
    o->beta = 0.4;
    o->frame_stack = 1;
    o->action_bytes = 4;
    o->ragged = 0;
    o->aux_elem_bytes = 0;
    o->payload_placement = CONDUIT_PLACE_HBM;
    o->weight_norm = CONDUIT_WNORM_BATCH;
    o->single_stream = 0;
}

const char* conduit_last_error(void) { return g_last_error.c_str(); }

const char* conduit_version(void) { return "conduit-mi355x 0.1 (gfx950)"; }

size_t conduit_buffer_required_bytes(int64_t capacity, const int64_t* obs_shape, int32_t ndim, conduit_dtype obs_dtype,
                                     const conduit_buffer_opts* opts) {
    conduit_buffer_opts o;
    conduit_buffer_opts_default(&o);
    if (opts) o = *opts;
    Layout L;
    if (make_layout(capacity, obs_shape, ndim, obs_dtype, o, &L) != CONDUIT_OK) return 0;
    return L.total;
}

conduit_status conduit_buffer_create(int64_t capacity, const int64_t* obs_shape, int32_t ndim, conduit_dtype obs_dtype,
                                     const conduit_buffer_opts* opts, void* arena, size_t arena_bytes,
                                     conduit_buffer** out) {
    if (!out) return fail(CONDUIT_EINVAL, "out must not be NULL");
    *out = nullptr;
    conduit_buffer_opts o;
    conduit_buffer_opts_default(&o);
    if (opts) o = *opts;
    Layout L;
    conduit_status st = make_layout(capacity, obs_shape, ndim, obs_dtype, o, &L);
    if (st != CONDUIT_OK) return st;
    if (arena) {
        if (arena_bytes < L.total) return fail(CONDUIT_EINVAL, "arena smaller than conduit_buffer_required_bytes()");
        if (reinterpret_cast<uintptr_t>(arena) % kAlign) return fail(CONDUIT_EINVAL, "arena must be 256-byte aligned");
    }
    int slot = -1;
    st = err_slot_acquire(&slot);
    if (st != CONDUIT_OK) return st;

    conduit_buffer* b = new conduit_buffer();
    (void)hipGetDevice(&b->device);
    b->capacity = capacity;
    b->obs_dtype = obs_dtype;
    b->opts = o;
    b->layout = L;
    b->err_slot = slot;
    if (arena) {
        b->arena = static_cast<uint8_t*>(arena);
    } else {
        void* p = nullptr;
        hipError_t e = hipMalloc(&p, L.total);
        if (e != hipSuccess) {
            err_slot_release(slot);
            delete b;
            (void)hipGetLastError();
            return fail(CONDUIT_ENOMEM, std::string("hipMalloc of ") + std::to_string(L.total) + " bytes failed");
        }
        b->arena = static_cast<uint8_t*>(p);
        b->owns_arena = true;
    }
    uint8_t* A = b->arena;
    b->state = reinterpret_cast<DeviceState*>(A + L.off_state);
    if (L.host_payload) {
        // coherent pinned host memory mapped into the device's address space:
        // the kernels reach it across the host link, uncached in the L2s, so
        // no XCD ever holds a stale line of it
        void* hp = nullptr;
        hipError_t e = hipHostMalloc(&hp, L.host_obs + L.host_aux, hipHostMallocMapped | hipHostMallocCoherent);
        if (e != hipSuccess) {
            (void)hipGetLastError();
            conduit_buffer_destroy(b);
            return fail(CONDUIT_ENOMEM, std::string("hipHostMalloc of ") + std::to_string(L.host_obs + L.host_aux) +
                                            " bytes failed");
        }
        b->host_payload = static_cast<uint8_t*>(hp);
        void* dp = nullptr;
        e = hipHostGetDevicePointer(&dp, hp, 0);
        if (e != hipSuccess) {
            conduit_status r = hip_fail(e, "hipHostGetDevicePointer");
            conduit_buffer_destroy(b);
            return r;
        }
        b->obs = static_cast<uint8_t*>(dp);
        b->aux = (o.ragged && o.aux_elem_bytes) ? b->obs + L.host_obs : nullptr;
    } else {
        b->obs = A + L.off_obs;
        b->aux = (o.ragged && o.aux_elem_bytes) ? A + L.off_aux : nullptr;
    }
    b->action = o.action_bytes ? A + L.off_action : nullptr;
    b->reward = reinterpret_cast<float*>(A + L.off_reward);
    b->done = A + L.off_done;
    b->episode = reinterpret_cast<uint32_t*>(A + L.off_episode);
    b->step = reinterpret_cast<int32_t*>(A + L.off_step);
    b->length = o.ragged ? reinterpret_cast<int32_t*>(A + L.off_length) : nullptr;
    TreeView& T = b->tree;
    T.depth = L.depth;
    T.alpha_num = o.alpha_num;
    T.alpha_den = o.alpha_den;
    T.frac_bits = (32 * (o.alpha_den - o.alpha_num)) / o.alpha_den;
    if (T.frac_bits > 31) T.frac_bits = 31;
    for (int l = 0; l <= kMaxLevels; ++l) {
        T.nodes[l] = l <= L.depth ? L.nodes[l] : 0;
        T.level[l] = nullptr;
        T.lds_offset[l] = -1;
    }
    if (o.prioritized) {
        T.leaves = reinterpret_cast<uint32_t*>(A + L.off_leaves);
        for (int l = 1; l <= L.depth; ++l) T.level[l] = reinterpret_cast<uint64_t*>(A + L.off_level[l]);
        int used = 0;
        for (int l = L.depth; l >= 1; --l) {  // small levels accumulate in LDS during updates
            if (L.nodes[l] <= 1024 && used + L.nodes[l] <= 2048) {
                T.lds_offset[l] = used;
                used += (int)L.nodes[l];
            }
        }
    }
    // initial contents: empty tree, unwritten slots (step -1), state words
    hipError_t e = hipSuccess;
    if (o.prioritized) {
        e = launch_fill_u32(T.leaves, 0u, round64(capacity), nullptr);
        for (int l = 1; l <= L.depth && e == hipSuccess; ++l)
            e = launch_fill_u64(T.level[l], 0ull, round64(L.nodes[l]), nullptr);
    }
    if (e == hipSuccess) e = launch_fill_u32(b->episode, 0u, capacity, nullptr);
    if (e == hipSuccess) e = launch_fill_u32(reinterpret_cast<uint32_t*>(b->step), 0xffffffffu, capacity, nullptr);
    if (e == hipSuccess && b->length) e = launch_fill_u32(reinterpret_cast<uint32_t*>(b->length), 0u, capacity, nullptr);
    DeviceState init{1u, 0xffffffffu, 0u, 0u};
    if (e == hipSuccess) e = hipMemcpy(b->state, &init, sizeof(init), hipMemcpyHostToDevice);
    if (e == hipSuccess) e = hipDeviceSynchronize();
    if (e != hipSuccess) {
        conduit_status r = hip_fail(e, "buffer initialisation");
        conduit_buffer_destroy(b);
        return r;
    }
    *out = b;
    return CONDUIT_OK;
}

void conduit_buffer_destroy(conduit_buffer* b) {
    if (!b) return;
    {
        DeviceGuard g(b->device);
        (void)hipDeviceSynchronize();
        if (b->owns_arena && b->arena) (void)hipFree(b->arena);
        if (b->host_payload) (void)hipHostFree(b->host_payload);
    }
    err_slot_release(b->err_slot);
    delete b;
}

conduit_status conduit_buffer_get_info(const conduit_buffer* b, conduit_buffer_info* info) {
    if (!b || !info) return fail(CONDUIT_EINVAL, "NULL argument");
    std::memset(info, 0, sizeof(*info));
    info->capacity = b->capacity;
    info->row_bytes = b->layout.row_bytes;
    info->head = b->head;
    info->size = b->size;
    info->total = b->total;
    info->tree_depth = b->opts.prioritized ? b->layout.depth : 0;
    for (int l = 0; l <= b->layout.depth && l < 8; ++l) info->tree_nodes[l] = b->layout.nodes[l];
    info->arena_bytes = (int64_t)b->layout.total;
    info->obs_dtype = (int32_t)b->obs_dtype;
    info->prioritized = b->opts.prioritized;
    info->frame_stack = b->opts.frame_stack;
    info->action_bytes = b->opts.action_bytes;
    info->ragged = b->opts.ragged;
    info->aux_elem_bytes = b->opts.aux_elem_bytes;
    info->max_len = b->layout.max_len;
    return CONDUIT_OK;
}

conduit_status conduit_buffer_stats(conduit_buffer* b, int64_t* size, int64_t* head, uint64_t* total) {
    if (!b) return fail(CONDUIT_EINVAL, "NULL buffer");
    DeviceGuard g(b->device);
    // every call enqueued on the buffer's device has finished: the ring state
    // below is then the one the device-side columns hold
    hipError_t e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail(e, "device synchronise");
    if (size) *size = b->size;
    if (head) *head = b->head;
    if (total) *total = (uint64_t)b->total;
    return check_flags(b->err_slot);
}

// Validated kernel arguments of an ingest (n > 0) at the buffer's current head.
static conduit_status ingest_args(conduit_buffer* b, const conduit_transitions* t, IngestArgs* out) {
    const conduit_buffer_opts& o = b->opts;
    if (!t->obs) return fail(CONDUIT_EINVAL, "obs must not be NULL");
    if (reinterpret_cast<uintptr_t>(t->obs) % 4) return fail(CONDUIT_EINVAL, "obs must be 4-byte aligned");
    if (o.ragged && !t->offsets) return fail(CONDUIT_EINVAL, "ragged ingest needs offsets");
    if (o.ragged && t->src_elems < 0) return fail(CONDUIT_EINVAL, "ragged ingest needs src_elems >= 0");
    if (o.ragged && t->aux && reinterpret_cast<uintptr_t>(t->aux) % 4) return fail(CONDUIT_EINVAL, "aux must be 4-byte aligned");
    if (o.frame_stack > 1 && !o.single_stream && (!t->episode_id || !t->step))
        return fail(CONDUIT_EINVAL, "frame-stacking buffers need episode_id and step (or the single_stream option)");
    IngestArgs a{};
    a.obs = b->obs;
    a.aux = b->aux;
    a.action = b->action;
    a.reward = b->reward;
    a.done = b->done;
    a.episode = b->episode;
    a.step = b->step;
    a.length = b->length;
    a.capacity = b->capacity;
    a.row_bytes = b->layout.row_bytes;
    a.max_len = b->layout.max_len;
    a.elem_bytes = o.ragged ? 4 : 0;
    a.aux_elem_bytes = o.aux_elem_bytes;
    a.action_bytes = o.action_bytes;
    a.prioritized = o.prioritized;
    a.src_obs = static_cast<const uint8_t*>(t->obs);
    a.src_offsets = t->offsets;
    a.src_elems = o.ragged ? t->src_elems : 0;
    a.src_aux = static_cast<const uint8_t*>(t->aux);
    a.src_action = static_cast<const uint8_t*>(t->action);
    a.src_reward = t->reward;
    a.src_done = t->done;
    a.src_episode = t->episode_id;
    a.src_step = t->step;
    a.src_prio = o.prioritized ? t->prio : nullptr;
    a.n = t->n;
    a.head = b->head;
    a.total = b->total;
    a.derive = o.single_stream ? (t->episode_id ? 0 : kDeriveEpisode) | (t->step ? 0 : kDeriveStep) : 0;
    a.tree = b->tree;
    a.state = b->state;
    a.err = err_words(b->err_slot);
    *out = a;
    return CONDUIT_OK;
}

// the host-known ring state after n more transitions
static void advance_ring(conduit_buffer* b, int64_t n) {
    b->head = (b->head + n) % b->capacity;
    b->size = b->size + n < b->capacity ? b->size + n : b->capacity;
    b->total += n;
}

// Validated kernel arguments of a priority update (n > 0).
static conduit_status update_args(conduit_buffer* b, const int64_t* idx, const uint32_t* prio, int64_t n,
                                  UpdateArgs* out) {
    if (!b->opts.prioritized) return fail(CONDUIT_EINVAL, "buffer was created without priorities");
    if (!idx || !prio) return fail(CONDUIT_EINVAL, "idx and prio must not be NULL");
    UpdateArgs a{};
    a.tree = b->tree;
    a.idx = idx;
    a.prio = prio;
    a.n = n;
    a.size = b->size;
    a.state = b->state;
    a.err = err_words(b->err_slot);
    *out = a;
    return CONDUIT_OK;
}

conduit_status conduit_ingest(conduit_buffer* b, const conduit_transitions* t, void* stream) {
    if (!b || !t) return fail(CONDUIT_EINVAL, "NULL buffer or transitions");
    conduit_status st = check_flags(b->err_slot);
    if (st != CONDUIT_OK) return st;
    if (t->n < 0 || t->n > b->capacity) return fail(CONDUIT_EINVAL, "ingest n must be in [0, capacity]");
    if (t->n == 0) return CONDUIT_OK;
    IngestArgs a{};
    st = ingest_args(b, t, &a);
    if (st != CONDUIT_OK) return st;
    DeviceGuard g(b->device);
    hipError_t e = launch_derive_meta(a, static_cast<hipStream_t>(stream));
    if (e == hipSuccess) e = launch_ingest(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "ingest launch");
    advance_ring(b, t->n);
    return CONDUIT_OK;
}

conduit_status conduit_update_priorities(conduit_buffer* b, const int64_t* idx, const uint32_t* prio, int64_t n,
                                         void* stream) {
    if (!b) return fail(CONDUIT_EINVAL, "NULL buffer");
    conduit_status st = check_flags(b->err_slot);
    if (st != CONDUIT_OK) return st;
    if (!b->opts.prioritized) return fail(CONDUIT_EINVAL, "buffer was created without priorities");
    if (n < 0) return fail(CONDUIT_EINVAL, "n must be >= 0");
    if (n == 0) return CONDUIT_OK;
    UpdateArgs a{};
    st = update_args(b, idx, prio, n, &a);
    if (st != CONDUIT_OK) return st;
    DeviceGuard g(b->device);
    hipError_t e = launch_update(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "update launch");
    return CONDUIT_OK;
}

// ingests of at most this many rows take the fused launch (its tree pass runs
// in one workgroup)
constexpr int64_t kFusedIngestMaxRows = 4096;

conduit_status conduit_update_ingest(conduit_buffer* b, const int64_t* idx, const uint32_t* prio, int64_t n_update,
                                     const conduit_transitions* t, void* stream) {
    if (!b || !t) return fail(CONDUIT_EINVAL, "NULL buffer or transitions");
    conduit_status st = check_flags(b->err_slot);
    if (st != CONDUIT_OK) return st;
    if (!b->opts.prioritized) return fail(CONDUIT_EINVAL, "buffer was created without priorities");
    if (n_update < 0) return fail(CONDUIT_EINVAL, "n_update must be >= 0");
    if (t->n < 0 || t->n > b->capacity) return fail(CONDUIT_EINVAL, "ingest n must be in [0, capacity]");
    UpdateArgs u{};
    if (n_update > 0) {
        st = update_args(b, idx, prio, n_update, &u);
        if (st != CONDUIT_OK) return st;
    }
    IngestArgs a{};
    if (t->n > 0) {
        st = ingest_args(b, t, &a);
        if (st != CONDUIT_OK) return st;
    }
    DeviceGuard g(b->device);
    hipStream_t s = static_cast<hipStream_t>(stream);
    // derived episode/step columns first: the update does not read them
    hipError_t e = t->n > 0 ? launch_derive_meta(a, s) : hipSuccess;
    if (e == hipSuccess) {
        if (n_update > 0 && t->n > 0 && !b->opts.ragged && t->n <= kFusedIngestMaxRows) {
            e = launch_update_ingest(u, a, s);
        } else {  // the same two operations, one launch each
            if (n_update > 0) e = launch_update(u, s);
            if (e == hipSuccess && t->n > 0) e = launch_ingest(a, s);
        }
    }
    if (e != hipSuccess) return hip_fail(e, "update + ingest launch");
    advance_ring(b, t->n);
    return CONDUIT_OK;
}

// buffer-wide weight normalisation: the sampler folds the leaf minimum
static void set_leaf_min(const conduit_buffer* b, SampleArgs* a) {
    if (a->w_out && b->opts.weight_norm == CONDUIT_WNORM_BUFFER) {
        a->leaf_min = &b->state->leaf_min;
        a->leaves = b->tree.leaves;
        a->n_leaves4 = round64(b->capacity) / 4;
    }
}

conduit_status conduit_sample(conduit_buffer* b, int64_t batch, const uint64_t* uniforms, int64_t* idx_out,
                              float* is_w_out, void* stream) {
    if (!b) return fail(CONDUIT_EINVAL, "NULL buffer");
    conduit_status st = check_flags(b->err_slot);
    if (st != CONDUIT_OK) return st;
    if (!b->opts.prioritized) return fail(CONDUIT_EINVAL, "buffer was created without priorities");
    if (batch < 1 || batch > (1LL << 20)) return fail(CONDUIT_EINVAL, "batch must be in [1, 2^20]");
    if (!uniforms || !idx_out) return fail(CONDUIT_EINVAL, "uniforms and idx_out must not be NULL");
    if (b->size == 0) return fail(CONDUIT_EEMPTY, "sample from an empty buffer");
    DeviceGuard g(b->device);
    SampleArgs a{};
    a.tree = b->tree;
    a.uniforms = uniforms;
    a.idx_out = idx_out;
    a.w_out = is_w_out;
    a.batch = batch;
    a.beta = b->opts.beta;
    a.state = b->state;
    a.err = err_words(b->err_slot);
    set_leaf_min(b, &a);
    hipError_t e = launch_sample(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "sample launch");
    return CONDUIT_OK;
}

static conduit_status check_xform(const conduit_transform* xf, int64_t row_bytes, conduit_dtype dt) {
    switch (xf->kind) {
        case CONDUIT_XF_NONE:
            return CONDUIT_OK;
        case CONDUIT_XF_U8_F32:
            if (dt != CONDUIT_U8) return fail(CONDUIT_EINVAL, "U8_F32 needs uint8 observations");
            return CONDUIT_OK;
        case CONDUIT_XF_U8_BF16_NORM:
            if (dt != CONDUIT_U8) return fail(CONDUIT_EINVAL, "U8_BF16_NORM needs uint8 observations");
            if (xf->channels < 1 || xf->channels > 4) return fail(CONDUIT_EINVAL, "channels must be in [1, 4]");
            if (row_bytes % (4 * xf->channels)) return fail(CONDUIT_EINVAL, "row must split into 4-byte-aligned planes");
            for (int c = 0; c < xf->channels; ++c)
                if (!(xf->std[c] != 0.0f)) return fail(CONDUIT_EINVAL, "std must be non-zero");
            return CONDUIT_OK;
        default:
            return fail(CONDUIT_EINVAL, "unknown or unsupported transform");
    }
}

static void fill_norm(GatherArgs& a, const conduit_transform* xf, int64_t row_bytes) {
    if (xf->kind != CONDUIT_XF_U8_BF16_NORM) {
        a.plane_units = 1;
        return;
    }
    a.plane_units = (int32_t)(row_bytes / 4 / xf->channels);
    for (int c = 0; c < 4; ++c) {
        a.mean[c] = c < xf->channels ? xf->mean[c] : 0.0f;
        a.stdv[c] = c < xf->channels ? xf->std[c] : 1.0f;
    }
}

// Validate a learner-batch request against the buffer and fill the kernel
// arguments (dense: GatherArgs, ragged: PackArgs).
static conduit_status prepare_gather(conduit_buffer* b, const int64_t* idx, int64_t n, const conduit_transform* xf,
                                     const conduit_learner_batch* out, GatherArgs* ga, PackArgs* pa) {
    const conduit_buffer_opts& o = b->opts;
    if (o.ragged) {
        if (xf->kind != CONDUIT_XF_TOKENS_PAD) return fail(CONDUIT_EINVAL, "ragged buffers gather with TOKENS_PAD");
        if (!out->obs) return fail(CONDUIT_EINVAL, "obs output must not be NULL");
        if ((reinterpret_cast<uintptr_t>(out->obs) | reinterpret_cast<uintptr_t>(out->aux)) % 16)
            return fail(CONDUIT_EINVAL, "outputs must be 16-byte aligned");
        if (reinterpret_cast<uintptr_t>(out->mask) % 4) return fail(CONDUIT_EINVAL, "mask must be 4-byte aligned");
        PackArgs a{};
        a.idx = idx;
        a.n = n;
        a.size = b->size;
        a.seq = b->obs;
        a.aux = b->aux;
        a.length = b->length;
        a.reward = b->reward;
        a.max_len = b->layout.max_len;
        a.pad_id = xf->pad_id;
        a.out_seq = out->obs;
        a.out_mask = out->mask;
        a.out_aux = b->aux ? out->aux : nullptr;
        a.out_length = out->length;
        a.out_reward = out->reward;
        a.action = b->action;
        a.out_action = b->action ? static_cast<uint8_t*>(out->action) : nullptr;
        a.action_bytes = o.action_bytes;
        a.done = b->done;
        a.out_done = out->done;
        a.err = err_words(b->err_slot);
        *pa = a;
        return CONDUIT_OK;
    }
    conduit_status st = check_xform(xf, b->layout.row_bytes, b->obs_dtype);
    if (st != CONDUIT_OK) return st;
    if (reinterpret_cast<uintptr_t>(out->obs) % 16) return fail(CONDUIT_EINVAL, "obs output must be 16-byte aligned");
    GatherArgs a{};
    a.idx = idx;
    a.n = n;
    a.limit = b->size;
    a.stack = o.frame_stack;
    a.capacity = b->capacity;
    a.src = b->obs;
    a.row_bytes = b->layout.row_bytes;
    a.episode = b->episode;
    a.step = b->step;
    a.out = out->obs;
    a.xform = xf->kind;
    fill_norm(a, xf, b->layout.row_bytes);
    a.action = b->action;
    a.out_action = b->action ? static_cast<uint8_t*>(out->action) : nullptr;
    a.action_bytes = o.action_bytes;
    a.reward = b->reward;
    a.out_reward = out->reward;
    a.done = b->done;
    a.out_done = out->done;
    a.ncols = 0;
    a.err = err_words(b->err_slot);
    a.err_kind = ERR_GATHER_INDEX;
    *ga = a;
    return CONDUIT_OK;
}

conduit_status conduit_gather_transform(conduit_buffer* b, const int64_t* idx, int64_t n, const conduit_transform* xf,
                                        const conduit_learner_batch* out, void* stream) {
    if (!b || !xf || !out) return fail(CONDUIT_EINVAL, "NULL buffer, transform or output");
    conduit_status st = check_flags(b->err_slot);
    if (st != CONDUIT_OK) return st;
    if (n < 0) return fail(CONDUIT_EINVAL, "n must be >= 0");
    if (n == 0) return CONDUIT_OK;
    if (!idx) return fail(CONDUIT_EINVAL, "idx must not be NULL");
    GatherArgs ga{};
    PackArgs pa{};
    st = prepare_gather(b, idx, n, xf, out, &ga, &pa);
    if (st != CONDUIT_OK) return st;
    DeviceGuard g(b->device);
    hipError_t e = b->opts.ragged ? launch_pack(pa, static_cast<hipStream_t>(stream))
                                  : launch_gather(ga, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "gather launch");
    return CONDUIT_OK;
}

conduit_status conduit_sample_gather(conduit_buffer* b, int64_t batch, const uint64_t* uniforms, int64_t* idx_out,
                                     float* is_w_out, const conduit_transform* xf, const conduit_learner_batch* out,
                                     void* stream) {
    if (!b || !xf || !out) return fail(CONDUIT_EINVAL, "NULL buffer, transform or output");
    conduit_status st = check_flags(b->err_slot);
    if (st != CONDUIT_OK) return st;
    if (!b->opts.prioritized) return fail(CONDUIT_EINVAL, "buffer was created without priorities");
    if (batch < 1 || batch > (1LL << 20)) return fail(CONDUIT_EINVAL, "batch must be in [1, 2^20]");
    if (!uniforms || !idx_out) return fail(CONDUIT_EINVAL, "uniforms and idx_out must not be NULL");
    if (b->size == 0) return fail(CONDUIT_EEMPTY, "sample from an empty buffer");
    GatherArgs ga{};
    PackArgs pa{};
    st = prepare_gather(b, idx_out, batch, xf, out, &ga, &pa);
    if (st != CONDUIT_OK) return st;
    DeviceGuard g(b->device);
    SampleArgs sa{};
    sa.tree = b->tree;
    sa.uniforms = uniforms;
    sa.idx_out = idx_out;
    sa.w_out = is_w_out;
    sa.batch = batch;
    sa.beta = b->opts.beta;
    sa.state = b->state;
    sa.err = err_words(b->err_slot);
    set_leaf_min(b, &sa);
    hipStream_t s = static_cast<hipStream_t>(stream);
    // dense rows of a few work items, and ragged rows: one fused launch
    hipError_t e = b->opts.ragged ? launch_sample_pack(sa, pa, nullptr, s) : launch_sample_gather(sa, ga, s);
    if (e == hipErrorNotSupported) {
        // otherwise the sampler parks the sampled leaves in is_w_out, and the
        // gather (or packing) launch carries one more workgroup that turns them
        // into the IS weights
        const WeightsArgs wa{is_w_out, batch, b->opts.beta, sa.leaf_min};
        ga.weights = wa;
        pa.weights = wa;
        e = launch_descend(sa, s);
        if (e == hipSuccess) e = b->opts.ragged ? launch_pack(pa, s) : launch_gather(ga, s);
    }
    if (e != hipSuccess) return hip_fail(e, "sample_gather launch");
    return CONDUIT_OK;
}

conduit_status conduit_nstep(conduit_buffer* b, const int64_t* idx, int64_t batch, int32_t n, double gamma,
                             int64_t* next_idx, float* ret, float* discount, uint8_t* valid,
                             const conduit_transform* xf, void* next_obs, void* stream) {
    if (!b) return fail(CONDUIT_EINVAL, "NULL buffer");
    conduit_status st = check_flags(b->err_slot);
    if (st != CONDUIT_OK) return st;
    if (batch < 0 || batch > (1LL << 20)) return fail(CONDUIT_EINVAL, "batch must be in [0, 2^20]");
    if (n < 1 || n > 63) return fail(CONDUIT_EINVAL, "n must be in [1, 63]");
    if (!(gamma == gamma)) return fail(CONDUIT_EINVAL, "gamma must be a number");
    if (batch == 0) return CONDUIT_OK;
    if (!idx || !next_idx || !ret || !discount || !valid) return fail(CONDUIT_EINVAL, "NULL index or output");
    if (b->size == 0) return fail(CONDUIT_EEMPTY, "n-step targets from an empty buffer");
    GatherArgs ga{};
    if (next_obs) {
        if (b->opts.ragged) return fail(CONDUIT_EINVAL, "next-state stacks need a dense buffer");
        if (!xf) return fail(CONDUIT_EINVAL, "next_obs needs a transform");
        conduit_learner_batch nb{};
        nb.obs = next_obs;
        PackArgs pa{};
        st = prepare_gather(b, next_idx, batch, xf, &nb, &ga, &pa);
        if (st != CONDUIT_OK) return st;
        ga.err_kind = -1;  // -1 entries are samples without a bootstrap state
    }
    DeviceGuard g(b->device);
    NstepArgs a{};
    a.idx = idx;
    a.batch = batch;
    a.n = n;
    a.gamma = gamma;
    a.capacity = b->capacity;
    a.size = b->size;
    a.total = b->total;
    a.reward = b->reward;
    a.done = b->done;
    a.episode = b->episode;
    a.next_idx = next_idx;
    a.ret = ret;
    a.discount = discount;
    a.valid = valid;
    a.err = err_words(b->err_slot);
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = next_obs ? launch_nstep_gather(a, ga, s) : hipErrorNotSupported;
    if (e == hipErrorNotSupported) {  // the targets, then the stacks: one launch each
        e = launch_nstep(a, s);
        if (e == hipSuccess && next_obs) e = launch_gather(ga, s);
    }
    if (e != hipSuccess) return hip_fail(e, "nstep launch");
    return CONDUIT_OK;
}

conduit_status conduit_sample_gather_nstep(conduit_buffer* b, int64_t batch, const uint64_t* uniforms,
                                           int64_t* idx_out, float* is_w_out, const conduit_transform* xf,
                                           const conduit_learner_batch* out, int32_t n, double gamma,
                                           int64_t* next_idx, float* ret, float* discount, uint8_t* valid,
                                           void* next_obs, void* stream) {
    if (!b || !xf || !out) return fail(CONDUIT_EINVAL, "NULL buffer, transform or output");
    conduit_status st = check_flags(b->err_slot);
    if (st != CONDUIT_OK) return st;
    if (!b->opts.prioritized) return fail(CONDUIT_EINVAL, "buffer was created without priorities");
    if (batch < 1 || batch > (1LL << 20)) return fail(CONDUIT_EINVAL, "batch must be in [1, 2^20]");
    if (!uniforms || !idx_out) return fail(CONDUIT_EINVAL, "uniforms and idx_out must not be NULL");
    if (n < 1 || n > 63) return fail(CONDUIT_EINVAL, "n must be in [1, 63]");
    if (!(gamma == gamma)) return fail(CONDUIT_EINVAL, "gamma must be a number");
    if (!next_idx || !ret || !discount || !valid) return fail(CONDUIT_EINVAL, "NULL n-step output");
    if (next_obs && b->opts.ragged) return fail(CONDUIT_EINVAL, "next-state stacks need a dense buffer");
    if (b->size == 0) return fail(CONDUIT_EEMPTY, "sample from an empty buffer");
    GatherArgs ga{};
    PackArgs pa{};
    st = prepare_gather(b, idx_out, batch, xf, out, &ga, &pa);
    if (st != CONDUIT_OK) return st;
    if (next_obs) {  // the bootstrap stacks are laid out as a gather's obs output
        conduit_learner_batch nb{};
        nb.obs = next_obs;
        GatherArgs gn{};
        PackArgs pn{};
        st = prepare_gather(b, next_idx, batch, xf, &nb, &gn, &pn);
        if (st != CONDUIT_OK) return st;
    }
    if (!b->opts.ragged) {
        DeviceGuard g(b->device);
        SampleArgs sa{};
        sa.tree = b->tree;
        sa.uniforms = uniforms;
        sa.idx_out = idx_out;
        sa.w_out = is_w_out;
        sa.batch = batch;
        sa.beta = b->opts.beta;
        sa.state = b->state;
        sa.err = err_words(b->err_slot);
        set_leaf_min(b, &sa);
        NstepArgs na{};
        na.idx = idx_out;
        na.batch = batch;
        na.n = n;
        na.gamma = gamma;
        na.capacity = b->capacity;
        na.size = b->size;
        na.total = b->total;
        na.reward = b->reward;
        na.done = b->done;
        na.episode = b->episode;
        na.next_idx = next_idx;
        na.ret = ret;
        na.discount = discount;
        na.valid = valid;
        na.err = err_words(b->err_slot);
        const hipError_t e = launch_sample_gather_nstep(sa, ga, na, next_obs, static_cast<hipStream_t>(stream));
        if (e == hipSuccess) return CONDUIT_OK;
        if (e != hipErrorNotSupported) return hip_fail(e, "sample_gather_nstep launch");
    }
    // other shapes: the two calls
    st = conduit_sample_gather(b, batch, uniforms, idx_out, is_w_out, xf, out, stream);
    if (st != CONDUIT_OK) return st;
    return conduit_nstep(b, idx_out, batch, n, gamma, next_idx, ret, discount, valid, xf, next_obs, stream);
}

conduit_status conduit_sample_pack_gae(conduit_buffer* b, int64_t batch, const uint64_t* uniforms, int64_t* idx_out,
                                      float* is_w_out, const conduit_transform* xf, const conduit_learner_batch* out,
                                      const float* values, double gamma, double lambda, float* adv, float* ret,
                                      void* stream) {
    if (!b || !xf || !out) return fail(CONDUIT_EINVAL, "NULL buffer, transform or output");
    conduit_status st = check_flags(b->err_slot);
    if (st != CONDUIT_OK) return st;
    if (!b->opts.prioritized) return fail(CONDUIT_EINVAL, "buffer was created without priorities");
    if (!b->opts.ragged) return fail(CONDUIT_EINVAL, "packing needs a ragged buffer");
    if (batch < 1 || batch > (1LL << 20)) return fail(CONDUIT_EINVAL, "batch must be in [1, 2^20]");
    if (!uniforms || !idx_out) return fail(CONDUIT_EINVAL, "uniforms and idx_out must not be NULL");
    if (!out->reward || !out->length) return fail(CONDUIT_EINVAL, "the GAE reads the packed rewards and lengths");
    if (!adv || !ret) return fail(CONDUIT_EINVAL, "adv and ret must not be NULL");
    if (!(gamma == gamma) || !(lambda == lambda)) return fail(CONDUIT_EINVAL, "gamma/lambda must be numbers");
    if (b->size == 0) return fail(CONDUIT_EEMPTY, "sample from an empty buffer");
    GatherArgs ga_unused{};
    PackArgs pa{};
    st = prepare_gather(b, idx_out, batch, xf, out, &ga_unused, &pa);
    if (st != CONDUIT_OK) return st;
    DeviceGuard g(b->device);
    SampleArgs sa{};
    sa.tree = b->tree;
    sa.uniforms = uniforms;
    sa.idx_out = idx_out;
    sa.w_out = is_w_out;
    sa.batch = batch;
    sa.beta = b->opts.beta;
    sa.state = b->state;
    sa.err = err_words(b->err_slot);
    set_leaf_min(b, &sa);
    const GaePackedArgs gp{out->reward, out->length, values, batch, b->layout.max_len, gamma, lambda,
                           adv, ret, err_words(b->err_slot)};
    const hipError_t e = launch_sample_pack(sa, pa, &gp, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "sample_pack_gae launch");
    return CONDUIT_OK;
}

// true if [a, a + na) and [b, b + nb) share a byte (NULL ranges share none)
static bool overlaps(const void* a, int64_t na, const void* b, int64_t nb) {
    if (!a || !b) return false;
    const uintptr_t x = reinterpret_cast<uintptr_t>(a), y = reinterpret_cast<uintptr_t>(b);
    return x < y + (uintptr_t)nb && y < x + (uintptr_t)na;
}

// GAE outputs (adv, ret: T*E floats) may overlap neither each other nor any input
static bool gae_outputs_overlap(const float* rewards, const float* values, const uint8_t* dones,
                                const uint8_t* truncated, const float* final_values, const float* bootstrap,
                                int64_t T, int64_t E, const float* adv, const float* ret) {
    const int64_t nf = T * E * 4, nb = T * E;
    for (const float* o : {adv, ret}) {
        if (overlaps(o, nf, rewards, nf) || overlaps(o, nf, values, nf) || overlaps(o, nf, dones, nb) ||
            overlaps(o, nf, truncated, nb) || overlaps(o, nf, final_values, nf) || overlaps(o, nf, bootstrap, E * 4))
            return true;
    }
    return overlaps(adv, nf, ret, nf);
}

conduit_status conduit_gae(const float* rewards, const float* values, const uint8_t* dones, const float* bootstrap,
                           int64_t T, int64_t E, double gamma, double lambda, float* adv, float* ret, void* stream) {
    if (T < 0 || E < 0) return fail(CONDUIT_EINVAL, "T and E must be >= 0");
    if (E > kGaeMaxEnvs) return fail(CONDUIT_EINVAL, "E must be at most 2^19 environments");
    if (T == 0 || E == 0) return CONDUIT_OK;
    if (!rewards || !dones || !adv || !ret) return fail(CONDUIT_EINVAL, "rewards, dones, adv and ret must not be NULL");
    if (!(gamma == gamma) || !(lambda == lambda)) return fail(CONDUIT_EINVAL, "gamma/lambda must be numbers");
    if (gae_outputs_overlap(rewards, values, dones, nullptr, nullptr, bootstrap, T, E, adv, ret))
        return fail(CONDUIT_EINVAL, "adv and ret must overlap neither each other nor the inputs");
    conduit_status st = standalone_flags();
    if (st != CONDUIT_OK) return st;
    GaeArgs a{rewards, values, dones, bootstrap, T, E, gamma, lambda, adv, ret, nullptr, nullptr, err_words(0)};
    hipError_t e = launch_gae(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "gae launch");
    return CONDUIT_OK;
}

conduit_status conduit_gae_noalloc(const float* rewards, const float* values, const uint8_t* dones,
                                   const float* bootstrap, int64_t T, int64_t E, double gamma, double lambda,
                                   float* adv, float* ret, void* stream) {
    if (T < 0 || E < 0) return fail(CONDUIT_EINVAL, "T and E must be >= 0");
    if (E > kGaeMaxEnvs) return fail(CONDUIT_EINVAL, "E must be at most 2^19 environments");
    if (T == 0 || E == 0) return CONDUIT_OK;
    if (!rewards || !dones || !adv || !ret) return fail(CONDUIT_EINVAL, "rewards, dones, adv and ret must not be NULL");
    if (!(gamma == gamma) || !(lambda == lambda)) return fail(CONDUIT_EINVAL, "gamma/lambda must be numbers");
    if (gae_outputs_overlap(rewards, values, dones, nullptr, nullptr, bootstrap, T, E, adv, ret))
        return fail(CONDUIT_EINVAL, "adv and ret must overlap neither each other nor the inputs");
    // the look-back path holds at most kLookMaxTiles tiles in the static table
    auto al = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
    const bool vec = E % 4 == 0 && al(rewards) && al(values) && al(bootstrap) && al(adv) && al(ret) &&
                     (reinterpret_cast<uintptr_t>(dones) & 3) == 0;
    const GaePlan p = plan_gae(T, E, vec);
    if (p.path == GAE_LOOK_BACK && p.groups * p.segments > kLookMaxTiles)
        return fail(CONDUIT_EINVAL, "rollout needs more look-back tiles than the static table holds (4,096)");
    uint32_t* err = nullptr;
    hipError_t e = gae_noalloc_err_words(&err);
    if (e != hipSuccess) return hip_fail(e, "look-back table address (hipGetSymbolAddress)");
    GaeArgs a{rewards, values, dones, bootstrap, T, E, gamma, lambda, adv, ret, nullptr, nullptr, err};
    e = launch_gae(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "gae launch");
    return CONDUIT_OK;
}

conduit_status conduit_gae_truncated(const float* rewards, const float* values, const uint8_t* dones,
                                     const uint8_t* truncated, const float* final_values, const float* bootstrap,
                                     int64_t T, int64_t E, double gamma, double lambda, float* adv, float* ret,
                                     void* stream) {
    if (T < 0 || E < 0) return fail(CONDUIT_EINVAL, "T and E must be >= 0");
    if (E > kGaeMaxEnvs) return fail(CONDUIT_EINVAL, "E must be at most 2^19 environments");
    if (T == 0 || E == 0) return CONDUIT_OK;
    if (!rewards || !dones || !truncated || !final_values || !adv || !ret)
        return fail(CONDUIT_EINVAL, "rewards, dones, truncated, final_values, adv and ret must not be NULL");
    if (!(gamma == gamma) || !(lambda == lambda)) return fail(CONDUIT_EINVAL, "gamma/lambda must be numbers");
    if (gae_outputs_overlap(rewards, values, dones, truncated, final_values, bootstrap, T, E, adv, ret))
        return fail(CONDUIT_EINVAL, "adv and ret must overlap neither each other nor the inputs");
    conduit_status st = standalone_flags();
    if (st != CONDUIT_OK) return st;
    GaeArgs a{rewards, values, dones, bootstrap, T, E, gamma, lambda, adv, ret, truncated, final_values,
              err_words(0)};
    hipError_t e = launch_gae(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "gae launch");
    return CONDUIT_OK;
}

conduit_status conduit_gae_plan(int64_t T, int64_t E, int32_t aligned, int32_t* path, int32_t* chunk) {
    if (T < 0 || E < 0) return fail(CONDUIT_EINVAL, "T and E must be >= 0");
    if (!path || !chunk) return fail(CONDUIT_EINVAL, "path and chunk must not be NULL");
    const GaePlan p = plan_gae(T, E, aligned != 0 && E % 4 == 0);
    *path = p.path;
    *chunk = p.chunk;
    return CONDUIT_OK;
}

conduit_status conduit_gae_packed(const float* last_reward, const int32_t* lengths, const float* values, int64_t B,
                                  int64_t Lmax, double gamma, double lambda, float* adv, float* ret, void* stream) {
    if (B < 0 || Lmax < 0) return fail(CONDUIT_EINVAL, "B and Lmax must be >= 0");
    if (B == 0 || Lmax == 0) return CONDUIT_OK;
    if (!last_reward || !lengths || !adv || !ret) return fail(CONDUIT_EINVAL, "NULL required pointer");
    if (!(gamma == gamma) || !(lambda == lambda)) return fail(CONDUIT_EINVAL, "gamma/lambda must be numbers");
    conduit_status st = standalone_flags();
    if (st != CONDUIT_OK) return st;
    GaePackedArgs a{last_reward, lengths, values, B, Lmax, gamma, lambda, adv, ret, err_words(0)};
    hipError_t e = launch_gae_packed(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "gae_packed launch");
    return CONDUIT_OK;
}

conduit_status conduit_minibatch_gather(const void* src, int64_t row_bytes, int64_t n_src, const int64_t* perm,
                                        int64_t n, const conduit_transform* xf, void* out, const float* const* cols,
                                        float* const* cols_out, int32_t ncols, void* stream) {
    if (!xf) return fail(CONDUIT_EINVAL, "NULL transform");
    if (n < 0 || n_src < 0 || row_bytes < 0) return fail(CONDUIT_EINVAL, "sizes must be >= 0");
    if (ncols < 0 || ncols > kMaxCols) return fail(CONDUIT_EINVAL, "ncols must be in [0, 8]");
    if (n == 0) return CONDUIT_OK;
    if (!perm) return fail(CONDUIT_EINVAL, "perm must not be NULL");
    if (row_bytes % 4) return fail(CONDUIT_EINVAL, "row_bytes must be a multiple of 4");
    if (out && (!src || reinterpret_cast<uintptr_t>(src) % 4))
        return fail(CONDUIT_EINVAL, "src must be non-NULL and 4-byte aligned");
    if (out && reinterpret_cast<uintptr_t>(out) % 16) return fail(CONDUIT_EINVAL, "out must be 16-byte aligned");
    if (ncols > 0 && (!cols || !cols_out)) return fail(CONDUIT_EINVAL, "column arrays must not be NULL");
    for (int c = 0; c < ncols; ++c)
        if (!cols[c] || !cols_out[c]) return fail(CONDUIT_EINVAL, "column pointers must not be NULL");
    if (xf->kind == CONDUIT_XF_TOKENS_PAD) return fail(CONDUIT_EINVAL, "TOKENS_PAD is for ragged buffers");
    conduit_status st = check_xform(xf, row_bytes, CONDUIT_U8);
    if (st != CONDUIT_OK) return st;
    st = standalone_flags();
    if (st != CONDUIT_OK) return st;
    GatherArgs a{};
    a.idx = perm;
    a.n = n;
    a.limit = n_src;
    a.stack = 1;
    a.capacity = n_src;
    a.src = static_cast<const uint8_t*>(src);
    a.row_bytes = row_bytes;
    a.out = row_bytes > 0 ? out : nullptr;
    a.xform = xf->kind;
    fill_norm(a, xf, row_bytes);
    a.ncols = ncols;
    for (int c = 0; c < ncols; ++c) {
        a.cols[c] = cols[c];
        a.cols_out[c] = cols_out[c];
    }
    a.err = err_words(0);
    a.err_kind = ERR_PERM_INDEX;
    hipError_t e = launch_gather(a, static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "minibatch gather launch");
    return CONDUIT_OK;
}

conduit_status conduit_buffer_read(const conduit_buffer* b, conduit_column col, int32_t level, int64_t offset,
                                   int64_t nbytes, void* dst, void* stream) {
    if (!b || !dst) return fail(CONDUIT_EINVAL, "NULL buffer or destination");
    uint8_t* base = nullptr;
    int64_t bytes = 0;
    conduit_status st = column_span(b, col, level, &base, &bytes);
    if (st != CONDUIT_OK) return st;
    if (!base || offset < 0 || nbytes < 0 || offset + nbytes > bytes) return fail(CONDUIT_EINVAL, "range outside the column");
    if (nbytes == 0) return CONDUIT_OK;
    DeviceGuard g(b->device);
    hipError_t e = hipMemcpyAsync(dst, base + offset, (size_t)nbytes, hipMemcpyDefault,
                                  static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "column copy");
    return CONDUIT_OK;
}

conduit_status conduit_buffer_checkpoint_bytes(const conduit_buffer* b, uint64_t* bytes) {
    if (!b || !bytes) return fail(CONDUIT_EINVAL, "NULL buffer or size pointer");
    conduit_ckpt_header h;
    ckpt_header(b, &h);
    *bytes = h.image_bytes;
    return CONDUIT_OK;
}

conduit_status conduit_buffer_checkpoint(const conduit_buffer* b, void* dst, uint64_t dst_bytes, void* stream) {
    if (!b || !dst) return fail(CONDUIT_EINVAL, "NULL buffer or destination");
    conduit_ckpt_header h;
    ckpt_header(b, &h);
    if (dst_bytes < h.image_bytes) return fail(CONDUIT_EINVAL, "destination smaller than the checkpoint image");
    DeviceGuard g(b->device);
    hipStream_t s = static_cast<hipStream_t>(stream);
    uint8_t* out = static_cast<uint8_t*>(dst);
    hipError_t e = hipMemcpyAsync(out, &h, sizeof(h), hipMemcpyDefault, s);
    for (uint32_t k = 0; k < h.n_sections && e == hipSuccess; ++k) {
        uint8_t* base = nullptr;
        int64_t n = 0;
        (void)column_span(b, (conduit_column)h.section[k].column, 0, &base, &n);
        e = hipMemcpyAsync(out + h.section[k].offset, base, (size_t)n, hipMemcpyDefault, s);
    }
    // the header copy reads this frame's `h`: wait before returning
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "checkpoint copy");
    return CONDUIT_OK;
}

conduit_status conduit_buffer_restore(conduit_buffer* b, const void* src, uint64_t src_bytes, void* stream) {
    if (!b || !src) return fail(CONDUIT_EINVAL, "NULL buffer or source");
    conduit_ckpt_header h;
    if (src_bytes < sizeof(h)) return fail(CONDUIT_EINVAL, "source smaller than a checkpoint header");
    DeviceGuard g(b->device);
    hipStream_t s = static_cast<hipStream_t>(stream);
    hipError_t e = hipMemcpyAsync(&h, src, sizeof(h), hipMemcpyDefault, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "checkpoint header copy");
    conduit_ckpt_header want;
    ckpt_header(b, &want);
    if (std::memcmp(h.magic, want.magic, sizeof(h.magic)) != 0) return fail(CONDUIT_EINVAL, "not a checkpoint image");
    if (h.version != want.version) return fail(CONDUIT_EINVAL, "unsupported checkpoint version");
    if (h.capacity != want.capacity || h.row_bytes != want.row_bytes || h.max_len != want.max_len ||
        h.obs_dtype != want.obs_dtype || h.prioritized != want.prioritized || h.alpha_num != want.alpha_num ||
        h.alpha_den != want.alpha_den || h.action_bytes != want.action_bytes || h.ragged != want.ragged ||
        h.aux_elem_bytes != want.aux_elem_bytes)
        return fail(CONDUIT_EINVAL, "checkpoint of a buffer with another layout (capacity, observation, "
                                    "prioritisation, alpha, action or ragged options differ)");
    if (h.image_bytes != want.image_bytes || h.n_sections != want.n_sections)
        return fail(CONDUIT_EINVAL, "checkpoint section table does not match this buffer");
    for (uint32_t k = 0; k < h.n_sections; ++k) {
        const conduit_ckpt_section& a = h.section[k];
        const conduit_ckpt_section& w = want.section[k];
        if (a.column != w.column || a.offset != w.offset || a.bytes != w.bytes)
            return fail(CONDUIT_EINVAL, "checkpoint section table does not match this buffer");
    }
    if (src_bytes < h.image_bytes) return fail(CONDUIT_EINVAL, "source smaller than the checkpoint image");
    const int64_t C = b->capacity;
    if (h.total > (uint64_t)INT64_MAX || h.size != ((int64_t)h.total < C ? (int64_t)h.total : C) ||
        h.head != (int64_t)(h.total % (uint64_t)C))
        return fail(CONDUIT_EINVAL, "checkpoint ring state is not one that ingestion reaches");
    const uint8_t* in = static_cast<const uint8_t*>(src);
    for (uint32_t k = 0; k < h.n_sections && e == hipSuccess; ++k) {
        uint8_t* base = nullptr;
        int64_t n = 0;
        (void)column_span(b, (conduit_column)h.section[k].column, 0, &base, &n);
        e = hipMemcpyAsync(base, in + h.section[k].offset, (size_t)n, hipMemcpyDefault, s);
    }
    if (e == hipSuccess && b->opts.prioritized) e = launch_tree_rebuild(b->tree, s);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    if (e != hipSuccess) return hip_fail(e, "checkpoint restore");
    b->head = h.head;
    b->size = h.size;
    b->total = (int64_t)h.total;
    return CONDUIT_OK;
}

conduit_status conduit_sync_check(const conduit_buffer* b, void* stream) {
    int slot = 0;
    if (b) {
        slot = b->err_slot;
        DeviceGuard g(b->device);
        hipError_t e = hipStreamSynchronize(static_cast<hipStream_t>(stream));
        if (e != hipSuccess) return hip_fail(e, "stream synchronise");
        return check_flags(slot);
    }
    hipError_t e = hipStreamSynchronize(static_cast<hipStream_t>(stream));
    if (e != hipSuccess) return hip_fail(e, "stream synchronise");
    conduit_status st = check_flags(0);
    if (st != CONDUIT_OK) return st;
    // the allocation-free GAE call's words, in the current GPU's static table
    uint32_t w[kErrKinds];
    e = gae_noalloc_read_errors(w);
    if (e != hipSuccess) return hip_fail(e, "reading the static error words");
    std::string msg;
    for (int k = 0; k < kErrKinds; ++k) {
        if (w[k]) {
            if (!msg.empty()) msg += "; ";
            msg += kErrText[k];
        }
    }
    if (msg.empty()) return CONDUIT_OK;
    return fail(CONDUIT_ESTATE, "device-side error flagged earlier (conduit_gae_noalloc): " + msg);
}

void conduit_clear_error(conduit_buffer* b) {
    if (!b) (void)gae_noalloc_clear_errors();
    std::lock_guard<std::mutex> lk(g_err_mu);
    if (!g_err_host) return;
    const int slot = b ? b->err_slot : 0;
    std::memset(g_err_host + slot * kErrKinds, 0, sizeof(uint32_t) * kErrKinds);
}

}  // extern "C"
