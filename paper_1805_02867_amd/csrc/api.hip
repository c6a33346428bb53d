// C-ABI of the library: argument validation, kernel choice and launches.
// Declarations and the contract of every entry point are in osoftmax.h.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include <mutex>

#include "kernels.h"
#include "osoftmax.h"

namespace {

constexpr int64_t kMaxDim = 2147483647;  // 2^31 - 1
constexpr int kMaxDevices = 64;

size_t elem_size(int dtype) { return dtype == OSM_BF16 ? 2 : 4; }
int elems_per_vec(int dtype) { return dtype == OSM_BF16 ? 8 : 4; }

// ------------------------------------------------------------ device state
// Scratch of the split kernels, cached per stream: work on one stream runs in
// order, so successive calls on a stream share a buffer without allocating;
// distinct streams get distinct buffers.
struct ScratchSlot {
    hipStream_t stream;
    void* ptr;
    size_t bytes;
};
constexpr int kScratchSlots = 64;
constexpr size_t kScratchMin = 256 * 1024;

// Fixed scratch of softmax_topk_ex_noalloc: one copy per device, held until
// the process ends.  In host code `scratch` names a host-side stand-in, not
// device memory: its device address is looked up once per device (with the
// device current) and kept in DeviceState::scratch_ptr, which is what every
// launch and copy uses.
constexpr size_t kNoAllocBytes = OSM_NOALLOC_SCRATCH_BYTES;
static __device__ __align__(256) unsigned char scratch[kNoAllocBytes];

// Clears n 32-bit words (a kernel rather than a memset, so that a captured
// graph replays it as an ordinary kernel node).
__global__ void zero_u32(uint32_t* p, int64_t n) {
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i < n) p[i] = 0u;
}

struct DeviceState {
    std::once_flag once;
    int cus = 0;
    void* scratch_ptr = nullptr;  // device address of `scratch` (null if the lookup failed)
    hipMemPool_t pool = nullptr;
    bool pool_ok = false;
    std::mutex mu;  // guards the scratch and counter tables
    ScratchSlot slots[kScratchSlots] = {};
    int nslots = 0;
    ScratchSlot cslots[kScratchSlots] = {};  // zeroed counter arrays, per stream
    int ncslots = 0;
};
DeviceState g_dev[kMaxDevices];

DeviceState* device_state(int* dev_out) {
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return nullptr;
    DeviceState& s = g_dev[dev];
    std::call_once(s.once, [&s, dev]() {
        int cus = 0;
        if (hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
            cus <= 0)
            cus = 256;
        s.cus = cus;
        void* sp = nullptr;
        if (hipGetSymbolAddress(&sp, HIP_SYMBOL(scratch)) == hipSuccess && sp) s.scratch_ptr = sp;
        // A library-owned stream-ordered pool keeps split-V scratch cheap to
        // allocate and free on any stream without touching the device's
        // default pool settings.
        hipMemPoolProps props = {};
        props.allocType = hipMemAllocationTypePinned;
        props.handleTypes = hipMemHandleTypeNone;
        props.location.type = hipMemLocationTypeDevice;
        props.location.id = dev;
        if (hipMemPoolCreate(&s.pool, &props) == hipSuccess) {
            uint64_t keep = UINT64_MAX;
            (void)hipMemPoolSetAttribute(s.pool, hipMemPoolAttrReleaseThreshold, &keep);
            s.pool_ok = true;
        }
        (void)hipGetLastError();
    });
    if (dev_out) *dev_out = dev;
    return &s;
}

// The scratch and counter tables are guarded by the device's mutex, and a
// call that uses a stream's buffers holds it from acquiring them until its
// last launch has been enqueued (`lk`, locked by the first acquire): calls
// from several host threads on one stream then enqueue their kernels whole,
// one call after another, so no call's launches land between another's on
// the same buffers, and a buffer is replaced (its old copy freed in stream
// order) only between calls.

// Slot of `stream` in `tab`, creating it if the table has room; null if full.
ScratchSlot* find_slot(ScratchSlot* tab, int* n, hipStream_t stream) {
    for (int i = 0; i < *n; ++i)
        if (tab[i].stream == stream) return &tab[i];
    if (*n >= kScratchSlots) return nullptr;
    ScratchSlot* slot = &tab[(*n)++];
    *slot = ScratchSlot{stream, nullptr, 0};
    return slot;
}

// Scratch of at least `bytes` for work enqueued on `stream`.  A stream's
// buffer grows by a stream-ordered allocation from the library pool (the old
// one is freed in stream order behind the work already enqueued) and is kept
// until osm_stream_release or the end of the process.  Once the table is
// full, a call gets a buffer of its own (*temp = true) that it frees in
// stream order after its launches.
int acquire_scratch(DeviceState* ds, std::unique_lock<std::mutex>& lk, hipStream_t stream,
                    size_t bytes, void** out, bool* temp) {
    if (!ds->pool_ok) return OSM_ENOMEM;
    if (!lk.owns_lock()) lk.lock();
    ScratchSlot* slot = find_slot(ds->slots, &ds->nslots, stream);
    *temp = slot == nullptr;
    if (slot && slot->bytes >= bytes) {
        *out = slot->ptr;
        return OSM_OK;
    }
    size_t want = bytes;
    if (slot) {
        want = bytes > 2 * slot->bytes ? bytes : 2 * slot->bytes;
        want = want > kScratchMin ? want : kScratchMin;
    }
    void* p = nullptr;
    if (hipMallocFromPoolAsync(&p, want, ds->pool, stream) != hipSuccess || !p) {
        (void)hipGetLastError();
        return OSM_ENOMEM;
    }
    if (slot) {
        if (slot->ptr) (void)hipFreeAsync(slot->ptr, stream);
        slot->ptr = p;
        slot->bytes = want;
    }
    *out = p;
    return OSM_OK;
}

// A zeroed array of at least `count` 32-bit counters for work enqueued on
// `stream`; the kernels that use it leave it zeroed.  A stream's array grows
// by a stream-ordered allocation, cleared in stream order by a fill kernel
// (not a memset, so that a call captured into a graph records a kernel
// node); once the table is full, a call gets an array of its own
// (*temp = true) to free after its launches.  Locking as acquire_scratch.
int acquire_counters(DeviceState* ds, std::unique_lock<std::mutex>& lk, hipStream_t stream,
                     size_t count, uint32_t** out, bool* temp) {
    if (!ds->pool_ok) return OSM_ENOMEM;
    if (!lk.owns_lock()) lk.lock();
    ScratchSlot* slot = find_slot(ds->cslots, &ds->ncslots, stream);
    *temp = slot == nullptr;
    const size_t bytes = count * 4;
    if (slot && slot->bytes >= bytes) {
        *out = static_cast<uint32_t*>(slot->ptr);
        return OSM_OK;
    }
    size_t want = bytes;
    if (slot) want = bytes > 2 * slot->bytes ? bytes : 2 * slot->bytes;
    void* p = nullptr;
    if (hipMallocFromPoolAsync(&p, want, ds->pool, stream) != hipSuccess || !p) {
        (void)hipGetLastError();
        return OSM_ENOMEM;
    }
    const int64_t words = (int64_t)(want / 4);
    hipLaunchKernelGGL(zero_u32, dim3((unsigned)((words + 255) / 256)), dim3(256), 0, stream,
                       static_cast<uint32_t*>(p), words);
    if (hipGetLastError() != hipSuccess) {
        (void)hipFreeAsync(p, stream);
        return OSM_EHIP;
    }
    if (slot) {
        if (slot->ptr) (void)hipFreeAsync(slot->ptr, stream);
        slot->ptr = p;
        slot->bytes = want;
    }
    *out = static_cast<uint32_t*>(p);
    return OSM_OK;
}

// Drops `stream`'s slot from `tab` (its buffer freed in stream order).
hipError_t release_slot(ScratchSlot* tab, int* n, hipStream_t stream) {
    hipError_t e = hipSuccess;
    for (int i = 0; i < *n; ++i) {
        if (tab[i].stream != stream) continue;
        if (tab[i].ptr) e = hipFreeAsync(tab[i].ptr, stream);
        tab[i] = tab[*n - 1];
        --*n;
        break;
    }
    return e;
}

// ------------------------------------------------------------- validation
bool overlaps(const void* a, size_t abytes, const void* b, size_t bbytes) {
    uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return a0 < b0 + bbytes && b0 < a0 + abytes;
}

bool aligned(const void* p, size_t a) { return ((uintptr_t)p % a) == 0; }

// Sizes, dtype and byte count of an N x V batch; false on any violation.
bool check_shape(int64_t N, int64_t V, int dtype, size_t* bytes) {
    if (N < 0 || N > kMaxDim || V < 1 || V > kMaxDim) return false;
    if (dtype != OSM_F32 && dtype != OSM_BF16) return false;
    // N, V < 2^31 and element size <= 4: the product is below 2^64
    *bytes = (size_t)N * (size_t)V * elem_size(dtype);
    return true;
}

int hip_status(hipError_t e) { return e == hipSuccess ? OSM_OK : OSM_EHIP; }

// ---------------------------------------------------------------- planning
struct Plan {
    int kernel;
    int64_t param;
};

Plan choose(int64_t N, int64_t V, int dtype, int cus) {
    const int64_t E = elems_per_vec(dtype);
    const int64_t nv = (V + E - 1) / E;  // 16-byte vectors per row
    // Short rows: a lane group per row, sized so each lane has ~2-4 vectors.
    if (nv <= 16) return {OSM_KERNEL_ROWS, 4};
    if (nv <= 32) return {OSM_KERNEL_ROWS, 8};
    if (nv <= 64) return {OSM_KERNEL_ROWS, 16};
    if (nv <= 128) return {OSM_KERNEL_ROWS, 32};
    if (nv <= 1024) return {OSM_KERNEL_ROWS, 64};
    // Long rows but too few of them to fill the chip: split each row, into
    // about four chunks per CU in all, six for the smallest batches (at 10
    // rows of 10^6: 19.5 us with six against 22.5 with four; at 64 or 256
    // rows four is as fast or faster).
    const int64_t want_blocks = (N <= 16 ? 6 : 4) * (int64_t)cus;
    if (N < 2 * (int64_t)cus && V >= 16384) {
        int64_t S = (want_blocks + N - 1) / N;
        int64_t s_cap = (V + 4095) / 4096;  // keep chunks >= 4096 elements
        if (S > s_cap) S = s_cap;
        if (S >= 2) return {OSM_KERNEL_SPLIT, S};
    }
    if (nv <= 2048) return {OSM_KERNEL_ROWS, 256};
    if (nv <= 4096) return {OSM_KERNEL_ROWS, 512};
    return {OSM_KERNEL_ROWS, 1024};
}

// Row-resident mode: the first (block, 16-byte vectors per lane) shape that
// holds the row's vectors; false if none does.  Smaller workgroups come
// first: with 16 vectors per lane (4 wavefronts per SIMD) a CU then holds two
// or four rows at once, so one row's loads overlap another's reduction.
struct ResShape {
    int block, r;
};
bool choose_resident(int64_t V, int dtype, int64_t block_req, ResShape* out) {
    const int64_t need = V / elems_per_vec(dtype);  // at least the row's whole vectors
    static const ResShape shapes[] = {{256, 4}, {256, 8}, {256, 16}, {512, 16}, {1024, 16}};
    for (const ResShape& c : shapes) {
        if (block_req && c.block != block_req) continue;
        if (need <= (int64_t)c.block * c.r) {
            *out = c;
            return true;
        }
    }
    return false;
}

bool team_ok(int64_t t) {
    return t == 4 || t == 8 || t == 16 || t == 32 || t == 64 || t == 128 || t == 256 ||
           t == 512 || t == 1024;
}

int run_softmax(const void* x, void* y, int64_t N, int64_t V, int dtype, int mode, int kernel,
                int64_t param, hipStream_t stream) {
    size_t bytes = 0;
    if (!check_shape(N, V, dtype, &bytes)) return OSM_EINVAL;
    if (mode != OSM_NAIVE && mode != OSM_SAFE && mode != OSM_ONLINE && mode != OSM_RESIDENT)
        return OSM_EINVAL;
    if (kernel != OSM_KERNEL_AUTO && kernel != OSM_KERNEL_ROWS && kernel != OSM_KERNEL_SPLIT)
        return OSM_EINVAL;
    if (mode == OSM_RESIDENT) {
        if (kernel == OSM_KERNEL_SPLIT ||
            (kernel == OSM_KERNEL_ROWS && param != 256 && param != 512 && param != 1024))
            return OSM_EINVAL;
    } else {
        if (kernel == OSM_KERNEL_ROWS && !team_ok(param)) return OSM_EINVAL;
        if (kernel == OSM_KERNEL_SPLIT && (param < 1 || param > kMaxDim)) return OSM_EINVAL;
    }
    if (N == 0) return OSM_OK;
    if (!x || !y) return OSM_EINVAL;
    const size_t es = elem_size(dtype);
    if (!aligned(x, es) || !aligned(y, es)) return OSM_EINVAL;
    if (overlaps(x, bytes, y, bytes)) return OSM_EINVAL;
    const bool vec = (((uintptr_t)x - (uintptr_t)y) % 16) == 0;
    if (mode == OSM_RESIDENT) {
        ResShape rs;
        if (!choose_resident(V, dtype, kernel == OSM_KERNEL_ROWS ? param : 0, &rs))
            return OSM_EUNSUPPORTED;
        return hip_status(
            osm::launch_softmax_resident(x, y, N, V, dtype, rs.block, rs.r, vec, stream));
    }

    int dev = 0;
    DeviceState* ds = device_state(&dev);
    if (!ds) return OSM_EHIP;
    Plan p = kernel == OSM_KERNEL_AUTO ? choose(N, V, dtype, ds->cus) : Plan{kernel, param};

    if (p.kernel == OSM_KERNEL_ROWS)
        return hip_status(osm::launch_softmax_rows(x, y, N, V, dtype, mode, (int)p.param, vec,
                                                   stream));

    // split-V: chunk = ceil(V / S) rounded up to whole 16-byte vectors
    const int64_t E = elems_per_vec(dtype);
    int64_t S = p.param;
    if (S > V) S = V;
    int64_t chunk = (V + S - 1) / S;
    chunk = (chunk + E - 1) / E * E;
    S = (V + chunk - 1) / chunk;  // drop chunks that would start past the row
    if (N * S > kMaxDim) return OSM_EINVAL;
    void* part = nullptr;
    bool temp = false;
    std::unique_lock<std::mutex> lk(ds->mu, std::defer_lock);  // held until the launches are in
    const int st = acquire_scratch(ds, lk, stream, (size_t)N * (size_t)S * 8, &part, &temp);
    if (st != OSM_OK) return st;
    hipError_t e = osm::launch_softmax_split(x, y, part, N, V, dtype, mode, S, chunk, vec,
                                             stream);
    hipError_t f = temp ? hipFreeAsync(part, stream) : hipSuccess;
    if (e != hipSuccess) return OSM_EHIP;
    return hip_status(f);
}

// Top-k plan: one wavefront per row once the batch alone can give every
// SIMD several wavefronts, or when rows are short (up to 1536 elements: a
// wavefront streams them in a step or two, and more wavefronts per row only
// add the barrier and the cross-wavefront merge); a small batch of long rows
// is split into chunks (a workgroup each, at most two workgroups per CU in
// all, at least two chunks a row: every chunk pays a fixed selection cost, so
// more, shorter chunks stop paying off early, and a third workgroup on a few
// CUs slows their chunks, which the rows then wait for: 10 x 4e6 top-5 took
// 34.5 us in 510 workgroups against 41.8 in 520); otherwise a workgroup (four
// wavefronts) per row.
//
// The chunk count is also capped so that a row's S * K partial keys fit the
// merge's single register batch (512 keys; a larger merge goes through the
// queue and its repeated selections: 4 x 10^6 top-5 took 20.8 us at 128
// chunks against 15.7 at 52).
Plan choose_topk(int64_t N, int64_t V, int K, int cus) {
    if (N >= 4 * (int64_t)cus || V <= 1536) return {OSM_KERNEL_ROWS, 64};
    if (N < 2 * (int64_t)cus && V >= 8192) {
        int64_t S = (2 * (int64_t)cus) / N;
        if (S < 2) S = 2;
        int64_t s_cap = V / 4096;  // keep chunks >= 4096 elements
        if (S > s_cap) S = s_cap;
        const int64_t k_cap = 512 / K;
        if (S > k_cap) S = k_cap;
        if (S >= 2) return {OSM_KERNEL_SPLIT, S};
    }
    return {OSM_KERNEL_ROWS, 256};
}

// One top-k pass of variant `var` over x (already validated).  noalloc: the
// split path's partials and row counters go to the device's fixed scratch
// array instead of the stream's pool buffers.
int launch_topk_pass(const void* x, float* vals, int32_t* idx, int64_t N, int64_t V, int K,
                     int dtype, int var, int kernel, int64_t param, DeviceState* ds,
                     hipStream_t stream, bool noalloc = false) {
    Plan p = kernel == OSM_KERNEL_AUTO ? choose_topk(N, V, K, ds->cus) : Plan{kernel, param};
    osm::TopkLaunch a{x, vals, idx, nullptr, N, V, K, 1, 1, V, stream};
    if (p.kernel == OSM_KERNEL_ROWS) {
        a.waves_per_row = (int)(p.param / 64);
        return hip_status(osm::launch_topk(a, dtype, var));
    }
    // split: chunk = ceil(V / S) rounded up to whole 16-byte vectors
    const int64_t E = elems_per_vec(dtype);
    int64_t S = p.param;
    if (S > V) S = V;
    int64_t chunk = (V + S - 1) / S;
    chunk = (chunk + E - 1) / E * E;
    S = (V + chunk - 1) / chunk;  // drop chunks that would start past the row
    if (N * S > kMaxDim) return OSM_EINVAL;
    if (S == 1) {  // one chunk is the whole row
        a.waves_per_row = 4;
        return hip_status(osm::launch_topk(a, dtype, var));
    }
    a.S = S;
    a.chunk = chunk;
    if (noalloc) {
        // partials first, then N row counters (256-byte aligned), cleared by a
        // fill kernel in stream order before the split kernel
        const size_t pb = (osm::topk_part_bytes(N, S, K) + 255) / 256 * 256;
        if (pb + (size_t)N * 4 > kNoAllocBytes) return OSM_ESCRATCH;
        if (!ds->scratch_ptr) return OSM_EHIP;
        a.part = ds->scratch_ptr;
        a.ctr = reinterpret_cast<uint32_t*>(static_cast<char*>(ds->scratch_ptr) + pb);
        const int64_t blocks = (N + 255) / 256;
        hipLaunchKernelGGL(zero_u32, dim3((unsigned)blocks), dim3(256), 0, stream, a.ctr, N);
        hipError_t e = hipGetLastError();
        if (e != hipSuccess) return OSM_EHIP;
        return hip_status(osm::launch_topk(a, dtype, var));
    }
    void* part = nullptr;
    bool temp = false;
    std::unique_lock<std::mutex> lk(ds->mu, std::defer_lock);  // held until the launch is in
    int st = acquire_scratch(ds, lk, stream, osm::topk_part_bytes(N, S, K), &part, &temp);
    if (st != OSM_OK) return st;
    a.part = part;
    // per-row chunk counters: each row's last chunk merges it in the same kernel
    bool ctemp = false;
    st = acquire_counters(ds, lk, stream, (size_t)N, &a.ctr, &ctemp);
    if (st != OSM_OK) {
        if (temp) (void)hipFreeAsync(part, stream);
        return st;
    }
    hipError_t e = osm::launch_topk(a, dtype, var);
    hipError_t f = temp ? hipFreeAsync(part, stream) : hipSuccess;
    hipError_t g = ctemp ? hipFreeAsync(a.ctr, stream) : hipSuccess;
    if (e != hipSuccess) return OSM_EHIP;
    if (f != hipSuccess) return hip_status(f);
    return hip_status(g);
}

bool topk_algo_ok(int algo) {
    return algo == OSM_TOPK_ONLINE_FUSED || algo == OSM_TOPK_SAFE_FUSED ||
           algo == OSM_TOPK_SAFE_UNFUSED || algo == OSM_TOPK_ONLINE_UNFUSED ||
           algo == OSM_TOPK_VALUES;
}

int run_topk(const void* x, void* y, float* vals, int32_t* idx, int64_t N, int64_t V, int K,
             int dtype, int algo, int kernel, int64_t param, hipStream_t stream,
             bool noalloc = false) {
    size_t bytes = 0;
    if (!check_shape(N, V, dtype, &bytes)) return OSM_EINVAL;
    if (K < 1 || K > OSM_TOPK_KMAX || (int64_t)K > V) return OSM_EINVAL;
    if (!topk_algo_ok(algo)) return OSM_EINVAL;
    const bool unfused = algo == OSM_TOPK_SAFE_UNFUSED || algo == OSM_TOPK_ONLINE_UNFUSED;
    if (kernel == OSM_KERNEL_ROWS) {
        // the two-wavefront shape exists for the one-pass variant only
        const bool two_ok = algo == OSM_TOPK_ONLINE_FUSED;
        if (!(param == 64 || (param == 128 && two_ok) || param == 256)) return OSM_EINVAL;
    } else if (kernel == OSM_KERNEL_SPLIT) {
        if (param < 1 || param > kMaxDim || N * (param < V ? param : V) > kMaxDim)
            return OSM_EINVAL;
    } else if (kernel != OSM_KERNEL_AUTO) {
        return OSM_EINVAL;
    }
    if (N == 0) return OSM_OK;
    if (!x || !vals || !idx || (unfused && !y)) return OSM_EINVAL;
    const size_t es = elem_size(dtype);
    if (!aligned(x, es) || !aligned(vals, 4) || !aligned(idx, 4)) return OSM_EINVAL;
    const size_t ob = (size_t)N * (size_t)K * 4;
    if (overlaps(x, bytes, vals, ob) || overlaps(x, bytes, idx, ob) || overlaps(vals, ob, idx, ob))
        return OSM_EINVAL;
    if (unfused && (!aligned(y, es) || overlaps(y, bytes, x, bytes) ||
                    overlaps(y, bytes, vals, ob) || overlaps(y, bytes, idx, ob)))
        return OSM_EINVAL;
    DeviceState* ds = device_state(nullptr);
    if (!ds) return OSM_EHIP;
    switch (algo) {
        case OSM_TOPK_ONLINE_FUSED:
            return launch_topk_pass(x, vals, idx, N, V, K, dtype, osm::TK_ONLINE, kernel, param,
                                    ds, stream, noalloc);
        case OSM_TOPK_SAFE_FUSED:
            return launch_topk_pass(x, vals, idx, N, V, K, dtype, osm::TK_SAFE, kernel, param, ds,
                                    stream);
        case OSM_TOPK_VALUES:
            return launch_topk_pass(x, vals, idx, N, V, K, dtype, osm::TK_VALUES, kernel, param,
                                    ds, stream);
        default: {
            // softmax into y (Alg. 2 or Alg. 3), then a separate top-k over y
            const int mode = algo == OSM_TOPK_SAFE_UNFUSED ? OSM_SAFE : OSM_ONLINE;
            int st = run_softmax(x, y, N, V, dtype, mode, OSM_KERNEL_AUTO, 0, stream);
            if (st != OSM_OK) return st;
            return launch_topk_pass(y, vals, idx, N, V, K, dtype, osm::TK_VALUES, kernel, param,
                                    ds, stream);
        }
    }
}

// ---------------------------------------------------------------- projection
constexpr int64_t kProjTile = 128;     // smallest tile edge of the projection kernels
constexpr int64_t kProjMaxH = 1 << 20;  // 32-bit load offsets within a tile

// Arguments shared by the projection entry points; OSM_OK if valid.
int check_proj(const void* h, const void* w, int64_t N, int64_t H, int64_t V) {
    // the tile grid is one-dimensional: (N / 128) * (V / 128) workgroups < 2^31
    if (N < 0 || N > 65535 * kProjTile || V < 1 || V > kMaxDim || H < 8 || H > kProjMaxH ||
        H % 8 != 0 ||
        ((N + kProjTile - 1) / kProjTile) * ((V + kProjTile - 1) / kProjTile) > (kMaxDim - 7))
        return OSM_EINVAL;
    if (N == 0) return OSM_OK;
    if (!h || !w || !aligned(h, 16) || !aligned(w, 16)) return OSM_EINVAL;
    return OSM_OK;
}

int run_proj_logits(const void* h, const void* w, float* out, int64_t N, int64_t H, int64_t V,
                    hipStream_t stream) {
    int st = check_proj(h, w, N, H, V);
    if (st != OSM_OK || N == 0) return st;
    if (!out || !aligned(out, 4)) return OSM_EINVAL;
    const size_t ob = (size_t)N * (size_t)V * 4, hb = (size_t)N * (size_t)H * 2,
                 wb = (size_t)V * (size_t)H * 2;
    if (overlaps(out, ob, h, hb) || overlaps(out, ob, w, wb)) return OSM_EINVAL;
    DeviceState* ds = device_state(nullptr);
    if (!ds) return OSM_EHIP;
    return hip_status(osm::launch_proj_logits(h, w, out, N, H, V, ds->cus, stream));
}

int run_proj_topk(const void* h, const void* w, float* vals, int32_t* idx, int64_t N, int64_t H,
                  int64_t V, int K, hipStream_t stream) {
    int st = check_proj(h, w, N, H, V);
    if (st != OSM_OK) return st;
    if (K < 1 || K > OSM_PROJ_KMAX || (int64_t)K > V) return OSM_EINVAL;
    if (N == 0) return OSM_OK;
    if (!vals || !idx || !aligned(vals, 4) || !aligned(idx, 4)) return OSM_EINVAL;
    const size_t ob = (size_t)N * (size_t)K * 4, hb = (size_t)N * (size_t)H * 2,
                 wb = (size_t)V * (size_t)H * 2;
    if (overlaps(vals, ob, idx, ob) || overlaps(vals, ob, h, hb) || overlaps(vals, ob, w, wb) ||
        overlaps(idx, ob, h, hb) || overlaps(idx, ob, w, wb))
        return OSM_EINVAL;
    DeviceState* ds = device_state(nullptr);
    if (!ds) return OSM_EHIP;
    int64_t S = 1, tiles = 1;
    int parts = 2;
    osm::proj_topk_shape(N, V, K, ds->cus, &S, &tiles, &parts);
    void* part = nullptr;
    bool temp = false;
    std::unique_lock<std::mutex> lk(ds->mu, std::defer_lock);  // held until the launches are in
    st = acquire_scratch(ds, lk, stream, osm::proj_topk_part_bytes(N, S, parts, K), &part,
                         &temp);
    if (st != OSM_OK) return st;
    hipError_t e =
        osm::launch_proj_topk(h, w, vals, idx, part, N, H, V, K, S, tiles, parts, stream);
    hipError_t f = temp ? hipFreeAsync(part, stream) : hipSuccess;
    if (e != hipSuccess) return OSM_EHIP;
    return hip_status(f);
}

}  // namespace

extern "C" {

int softmax_fwd(const void* x, void* y, int64_t N, int64_t V, int dtype, int mode,
                hipStream_t stream) {
    return run_softmax(x, y, N, V, dtype, mode, OSM_KERNEL_AUTO, 0, stream);
}

int softmax_fwd_ex(const void* x, void* y, int64_t N, int64_t V, int dtype, int mode, int kernel,
                   int64_t param, hipStream_t stream) {
    return run_softmax(x, y, N, V, dtype, mode, kernel, param, stream);
}

int softmax_topk(const float* x, float* vals, int32_t* idx, int64_t N, int64_t V, int K,
                 hipStream_t stream) {
    return run_topk(x, nullptr, vals, idx, N, V, K, OSM_F32, OSM_TOPK_ONLINE_FUSED,
                    OSM_KERNEL_AUTO, 0, stream);
}

int softmax_topk_dt(const void* x, float* vals, int32_t* idx, int64_t N, int64_t V, int K,
                    int dtype, hipStream_t stream) {
    return run_topk(x, nullptr, vals, idx, N, V, K, dtype, OSM_TOPK_ONLINE_FUSED,
                    OSM_KERNEL_AUTO, 0, stream);
}

int softmax_topk_ex(const void* x, float* vals, int32_t* idx, int64_t N, int64_t V, int K,
                    int dtype, int kernel, int64_t param, hipStream_t stream) {
    return run_topk(x, nullptr, vals, idx, N, V, K, dtype, OSM_TOPK_ONLINE_FUSED, kernel, param,
                    stream);
}

int softmax_topk_ex_noalloc(const void* x, float* vals, int32_t* idx, int64_t N, int64_t V,
                            int K, int dtype, int kernel, int64_t param, hipStream_t stream) {
    return run_topk(x, nullptr, vals, idx, N, V, K, dtype, OSM_TOPK_ONLINE_FUSED, kernel, param,
                    stream, true);
}

int softmax_topk_algo(const void* x, void* y, float* vals, int32_t* idx, int64_t N, int64_t V,
                      int K, int dtype, int algo, int kernel, int64_t param, hipStream_t stream) {
    return run_topk(x, y, vals, idx, N, V, K, dtype, algo, kernel, param, stream);
}

int topk_fwd(const void* x, float* vals, int32_t* idx, int64_t N, int64_t V, int K, int dtype,
             hipStream_t stream) {
    return run_topk(x, nullptr, vals, idx, N, V, K, dtype, OSM_TOPK_VALUES, OSM_KERNEL_AUTO, 0,
                    stream);
}

int osm_topk_plan(int64_t N, int64_t V, int dtype, int K, int* kernel, int64_t* param) {
    size_t bytes = 0;
    if (!check_shape(N, V, dtype, &bytes)) return OSM_EINVAL;
    if (K < 1 || K > OSM_TOPK_KMAX || (int64_t)K > V) return OSM_EINVAL;
    if (!kernel || !param) return OSM_EINVAL;
    DeviceState* ds = device_state(nullptr);
    Plan p = choose_topk(N, V, K, ds ? ds->cus : 256);
    *kernel = p.kernel;
    *param = p.param;
    return OSM_OK;
}

int osm_ref_stream(int op, const void* x, void* y, int64_t bytes, hipStream_t stream) {
    if ((op != 0 && op != 1) || bytes < 0 || bytes % 16 != 0) return OSM_EINVAL;
    if (bytes == 0) return OSM_OK;
    if (!x || !y || !aligned(x, 16) || !aligned(y, 16)) return OSM_EINVAL;
    if (op == 1 && overlaps(x, (size_t)bytes, y, (size_t)bytes)) return OSM_EINVAL;
    DeviceState* ds = device_state(nullptr);
    if (!ds) return OSM_EHIP;
    return hip_status(osm::launch_ref_stream(op, x, y, bytes / 16, ds->cus, stream));
}

int proj_fwd(const void* h, const void* w, float* logits, int64_t N, int64_t H, int64_t V,
             hipStream_t stream) {
    return run_proj_logits(h, w, logits, N, H, V, stream);
}

int proj_softmax_topk(const void* h, const void* w, float* vals, int32_t* idx, int64_t N,
                      int64_t H, int64_t V, int K, hipStream_t stream) {
    return run_proj_topk(h, w, vals, idx, N, H, V, K, stream);
}

int osm_stream_release(hipStream_t stream) {
    DeviceState* ds = device_state(nullptr);
    if (!ds) return OSM_EHIP;
    std::lock_guard<std::mutex> guard(ds->mu);
    const hipError_t e = release_slot(ds->slots, &ds->nslots, stream);
    const hipError_t f = release_slot(ds->cslots, &ds->ncslots, stream);
    if (e != hipSuccess || f != hipSuccess) {
        (void)hipGetLastError();
        return OSM_EHIP;
    }
    return OSM_OK;
}

int osm_plan(int64_t N, int64_t V, int dtype, int mode, int* kernel, int64_t* param) {
    size_t bytes = 0;
    if (!check_shape(N, V, dtype, &bytes)) return OSM_EINVAL;
    if (mode != OSM_NAIVE && mode != OSM_SAFE && mode != OSM_ONLINE && mode != OSM_RESIDENT)
        return OSM_EINVAL;
    if (!kernel || !param) return OSM_EINVAL;
    if (mode == OSM_RESIDENT) {
        ResShape rs;
        if (!choose_resident(V, dtype, 0, &rs)) return OSM_EUNSUPPORTED;
        *kernel = OSM_KERNEL_ROWS;
        *param = rs.block;
        return OSM_OK;
    }
    DeviceState* ds = device_state(nullptr);
    Plan p = choose(N, V, dtype, ds ? ds->cus : 256);
    *kernel = p.kernel;
    *param = p.param;
    return OSM_OK;
}

const char* osm_status_string(int status) {
    switch (status) {
        case OSM_OK: return "success";
        case OSM_EINVAL: return "invalid argument";
        case OSM_EUNSUPPORTED: return "unsupported configuration";
        case OSM_EHIP: return "HIP error while enqueuing work";
        case OSM_ENOMEM: return "scratch allocation failed";
        case OSM_ESCRATCH: return "needs more than the fixed no-allocation scratch";
        default: return "unknown status";
    }
}

}  // extern "C"
