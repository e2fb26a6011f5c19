// Host side of the C ABI declared in include/blockserve.h: argument and
// descriptor validation (before anything is enqueued), work-list construction,
// descriptor upload through a content-addressed ring of pinned/device slots,
// and kernel launches on the caller's stream.
#include <algorithm>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstring>
#include <functional>
#include <memory>
#include <mutex>
#include <queue>
#include <string>
#include <vector>

#include "bs_internal.h"
#include "bs_refresh.h"

using namespace bs;

namespace {

// Upload slots: the ring starts with kSlots and grows, instead of waiting for
// the device, while every slot is still read by queued work; only past
// kMaxSlots distinct descriptor sets in flight does a call wait for the
// least recently used one.
constexpr int kSlots = 16;
constexpr int kMaxSlots = 256;

// An upload slot holds one device blob (descriptors plus the work list derived
// from them) and the host key it was built from. The key is the small input
// the blob is a function of (call kind, shape parameters, descriptor bytes), so
// a repeated call (every denoising step of a block-cycle repeats its
// descriptors) finds its blob by comparing the key alone and neither rebuilds
// nor re-uploads anything.
struct Slot {
  void* d = nullptr;       // device copy of the blob
  void* h = nullptr;       // pinned staging copy (immutable while live)
  size_t cap = 0;
  std::vector<unsigned char> key;
  uint64_t hash = 0;
  int meta[6] = {0, 0, 0, 0, 0, 0};  // blob layout (offsets, counts) recorded at build time
  hipEvent_t ready = nullptr;  // recorded after the upload
  hipEvent_t done = nullptr;   // recorded after the last launch that read it
  hipStream_t stream = nullptr;
  uint64_t used = 0;           // tick of the last call that used it (LRU order)
  bool live = false;
};

thread_local std::string g_err;

uint64_t fnv1a(const void* p, size_t n) {
  const unsigned char* b = static_cast<const unsigned char*>(p);
  uint64_t h = 1469598103934665603ull;
  for (size_t i = 0; i < n; ++i) h = (h ^ b[i]) * 1099511628211ull;
  return h ^ n;
}

}  // namespace

// Phase timing of bs_mixed_state_step: kProfPhases + 1 events per step
// (before attention, after attention, after the row reductions, after selection).
constexpr int kProfPhases = BS_PROFILE_PHASES;
struct Prof {
  std::vector<hipEvent_t> ev;
  int cap = 0;     // steps the ring holds
  int used = 0;    // steps recorded since bs_profile_begin
  bool on = false;
};

// ---- static device memory of the allocation-free step
// The descriptors and attention work items of one call, then its decode
// partials. Each GPU the library runs on holds its own copy of the array
// until the process ends; host code reaches it only through the address
// hipGetSymbolAddress returns for that device.
constexpr size_t kStaticBlobBytes = size_t(512) << 10;
constexpr size_t kStaticPartBytes = (size_t(8) << 20) - kStaticBlobBytes;
constexpr int kStaticStages = 4;     // pinned host stages of a context (calls in flight before one waits)
static __device__ __align__(256) unsigned char scratch[kStaticBlobBytes + kStaticPartBytes];

struct StaticPath {
  void* scratch = nullptr;                       // this device's `scratch` (device address)
  void* stage[kStaticStages] = {};               // pinned host copies of a call's blob
  hipEvent_t copied[kStaticStages] = {};         // recorded after the copy out of each stage
  int next = 0;
  std::unique_ptr<AttnItem[]> tmp;               // the work-list interleave's temporary
};

struct bs_ctx {
  int device = 0;
  StaticPath stat;
  std::vector<std::unique_ptr<Slot>> slots;   // stable addresses: calls hold Slot*
  uint64_t tick = 0;
  std::string err;
  Prof prof;
};

namespace {

int fail(bs_ctx* c, int st, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  if (c)
    c->err = buf;
  else
    g_err = buf;
  return st;
}

int hip_fail(bs_ctx* c, hipError_t e, const char* what) {
  return fail(c, BS_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

// Makes the context's device current for the duration of a call.
struct DeviceGuard {
  int prev = -1;
  bool ok = true;
  explicit DeviceGuard(int dev) {
    if (hipGetDevice(&prev) != hipSuccess) prev = -1;
    if (prev != dev) ok = hipSetDevice(dev) == hipSuccess;
  }
  ~DeviceGuard() {
    int cur = -1;
    if (prev >= 0 && hipGetDevice(&cur) == hipSuccess && cur != prev) (void)hipSetDevice(prev);
  }
};

int check_reqs(bs_ctx* c, const bs_req_desc* reqs, int n, int L, int R, int W) {
  if (n < 0) return fail(c, BS_ERR_INVALID_ARG, "n < 0");
  if (n > 0 && !reqs) return fail(c, BS_ERR_INVALID_ARG, "reqs is NULL");
  if (L < 1) return fail(c, BS_ERR_DESCRIPTOR, "L < 1");
  if (R < 1 || W < 1) return fail(c, BS_ERR_INVALID_ARG, "box R=%d W=%d must be >= 1", R, W);
  std::vector<unsigned char> seen((size_t)R, 0);
  for (int i = 0; i < n; ++i) {
    const bs_req_desc& r = reqs[i];
    if (r.p < 0 || r.g < 1) return fail(c, BS_ERR_DESCRIPTOR, "request %d: p=%d g=%d (need p >= 0, g >= 1)", i, r.p, r.g);
    const int64_t K = ((int64_t)r.g + L - 1) / L;
    if (r.k < 0 || r.k >= K) return fail(c, BS_ERR_DESCRIPTOR, "request %d: block index %d outside [0, %lld)", i, r.k, (long long)K);
    if (r.row < 0 || r.row >= R) return fail(c, BS_ERR_DESCRIPTOR, "request %d: row %d outside [0, %d)", i, r.row, R);
    if (seen[r.row]) return fail(c, BS_ERR_DESCRIPTOR, "request %d: row %d used twice", i, r.row);
    seen[r.row] = 1;
    if (r.off < 0 || (int64_t)r.off + r.p + r.g > W)
      return fail(c, BS_ERR_DESCRIPTOR, "request %d: off=%d + p+g=%d exceeds W=%d", i, r.off, r.p + r.g, W);
  }
  return BS_OK;
}

bool aligned(const void* p, size_t a) { return (reinterpret_cast<uintptr_t>(p) % a) == 0; }

// Blob = descriptors followed by an optional work list, 16-byte aligned parts.
struct Blob {
  std::vector<unsigned char> bytes;
  int meta[6] = {0, 0, 0, 0, 0, 0};
  size_t add(const void* p, size_t n) {
    size_t off = (bytes.size() + 15) & ~size_t(15);
    bytes.resize(off + n);
    if (n) std::memcpy(bytes.data() + off, p, n);
    return off;
  }
};

// Key of a call: a tag and shape parameters, followed by the descriptor bytes.
struct Key {
  std::vector<unsigned char> b;
  Key(char tag, std::initializer_list<int64_t> params, const void* data, size_t n) {
    b.push_back(static_cast<unsigned char>(tag));
    for (int64_t v : params) push(&v, sizeof v);
    push(data, n);
  }
  void push(const void* p, size_t n) {
    const unsigned char* q = static_cast<const unsigned char*>(p);
    b.insert(b.end(), q, q + n);
  }
};

// Slot for a new blob: a new one while the ring holds fewer than kSlots
// (that many blobs stay cached); then the least recently used slot that no
// queued work still reads; a new slot while none is free and the ring is
// below kMaxSlots; otherwise (more than kMaxSlots descriptor sets in flight)
// the least recently used slot after waiting for its last reader -- the one
// bounded host wait.
int take_slot(bs_ctx* c, Slot** out) {
  if (c->slots.size() < (size_t)kSlots) {
    c->slots.push_back(std::make_unique<Slot>());
    *out = c->slots.back().get();
    return BS_OK;
  }
  Slot* lru_free = nullptr;
  Slot* lru_any = nullptr;
  for (auto& p : c->slots) {
    Slot* sl = p.get();
    if (!lru_any || sl->used < lru_any->used) lru_any = sl;
    bool free_ = !sl->live;
    if (!free_) {
      const hipError_t q = hipEventQuery(sl->done);
      if (q == hipSuccess)
        free_ = true;
      else if (q != hipErrorNotReady)
        return hip_fail(c, q, "hipEventQuery(slot)");
    }
    if (free_ && (!lru_free || sl->used < lru_free->used)) lru_free = sl;
  }
  Slot* sl = lru_free;
  if (!sl && c->slots.size() < (size_t)kMaxSlots) {
    c->slots.push_back(std::make_unique<Slot>());
    sl = c->slots.back().get();
  }
  if (!sl) {
    sl = lru_any;
    hipError_t e = hipEventSynchronize(sl->done);
    if (e != hipSuccess) return hip_fail(c, e, "hipEventSynchronize(slot)");
  }
  sl->live = false;
  *out = sl;
  return BS_OK;
}

// Find the slot built from `key`, or build the blob with make(Blob&) and
// upload it into a slot no queued work reads (take_slot).
template <class Make>
int upload(bs_ctx* c, hipStream_t s, const Key& key, Make make, Slot** out) {
  const uint64_t hv = fnv1a(key.b.data(), key.b.size());
  ++c->tick;
  for (auto& p : c->slots) {
    Slot& sl = *p;
    if (sl.live && sl.hash == hv && sl.key == key.b) {
      if (sl.stream != s) {
        hipError_t e = hipStreamWaitEvent(s, sl.done, 0);
        if (e != hipSuccess) return hip_fail(c, e, "hipStreamWaitEvent");
        sl.stream = s;
      }
      sl.used = c->tick;
      *out = &sl;
      return BS_OK;
    }
  }
  Blob blob;
  make(blob);
  const size_t n = blob.bytes.size();
  Slot* slp = nullptr;
  int st = take_slot(c, &slp);
  if (st) return st;
  Slot& sl = *slp;
  sl.used = c->tick;
  if (sl.cap < n) {
    if (sl.d) (void)hipFree(sl.d);
    if (sl.h) (void)hipHostFree(sl.h);
    sl.d = sl.h = nullptr;
    sl.cap = 0;
    size_t cap = 65536;
    while (cap < n) cap *= 2;
    hipError_t e = hipMalloc(&sl.d, cap);
    if (e != hipSuccess) return hip_fail(c, e, "hipMalloc(upload slot)");
    e = hipHostMalloc(&sl.h, cap, hipHostMallocDefault);
    if (e != hipSuccess) return hip_fail(c, e, "hipHostMalloc(upload slot)");
    sl.cap = cap;
  }
  if (!sl.ready) {
    hipError_t e = hipEventCreateWithFlags(&sl.ready, hipEventDisableTiming);
    if (e == hipSuccess) e = hipEventCreateWithFlags(&sl.done, hipEventDisableTiming);
    if (e != hipSuccess) return hip_fail(c, e, "hipEventCreate");
  }
  std::memcpy(sl.h, blob.bytes.data(), n);
  hipError_t e = hipMemcpyAsync(sl.d, sl.h, n, hipMemcpyHostToDevice, s);
  if (e != hipSuccess) return hip_fail(c, e, "hipMemcpyAsync(upload)");
  e = hipEventRecord(sl.ready, s);
  if (e != hipSuccess) return hip_fail(c, e, "hipEventRecord");
  sl.key = key.b;
  sl.hash = hv;
  std::memcpy(sl.meta, blob.meta, sizeof sl.meta);
  sl.stream = s;
  sl.live = true;
  *out = &sl;
  return BS_OK;
}

// The request descriptors alone (gather, scatter, decode share this blob).
int upload_reqs(bs_ctx* c, hipStream_t s, const bs_req_desc* reqs, int n, Slot** out) {
  return upload(c, s, Key('R', {n}, reqs, sizeof(bs_req_desc) * n),
                [&](Blob& b) { b.add(reqs, sizeof(bs_req_desc) * n); }, out);
}

int finish(bs_ctx* c, Slot* sl, hipStream_t s, hipError_t launch, const char* what) {
  hipError_t e = hipEventRecord(sl->done, s);
  if (launch != hipSuccess) return hip_fail(c, launch, what);
  if (e != hipSuccess) return hip_fail(c, e, "hipEventRecord(done)");
  return BS_OK;
}

int dtype_bytes(bs_dtype dt) { return dt == BS_F32 ? 4 : (dt == BS_BF16 ? 2 : 0); }

// ---- attention helpers shared by the K2 entry point and the fused step
int check_attention(bs_ctx* c, int n, int L, int Hq, int Hkv, int D, bs_dtype dt) {
  (void)n;
  if (dt != BS_F32 && dt != BS_BF16) return fail(c, BS_ERR_INVALID_ARG, "bad dtype %d", (int)dt);
  if (Hq < 1 || Hkv < 1 || D < 1) return fail(c, BS_ERR_INVALID_ARG, "Hq, Hkv, D must be >= 1");
  if (Hq % Hkv) return fail(c, BS_ERR_UNSUPPORTED, "Hq=%d not a multiple of Hkv=%d", Hq, Hkv);
  const int G = Hq / Hkv, RB = (L + 31) / 32;
  if (dt == BS_F32 && (D % 4 || D > 256))
    return fail(c, BS_ERR_UNSUPPORTED, "fp32 path needs D %% 4 == 0 and D <= 256 (D=%d)", D);
  if (dt == BS_BF16) {
    if (D != 64 && D != 128) return fail(c, BS_ERR_UNSUPPORTED, "bf16 path needs D in {64, 128} (D=%d)", D);
    if (L > 64 || G > 8)
      return fail(c, BS_ERR_UNSUPPORTED, "bf16 path needs L <= 64 and Hq/Hkv <= 8 (L=%d, Hq/Hkv=%d)", L, G);
    (void)RB;
  }
  return BS_OK;
}

// layer < 0: the single-layer entry point (no layer in the message)
int check_attention_tensors(bs_ctx* c, const void* q, const void* k_new, const void* v_new, const void* k_cache,
                            const void* v_cache, const void* out, int layer) {
  if (!q || !k_new || !v_new || !k_cache || !v_cache || !out)
    return layer < 0 ? fail(c, BS_ERR_INVALID_ARG, "tensor pointer is NULL")
                     : fail(c, BS_ERR_INVALID_ARG, "layer %d: tensor pointer is NULL", layer);
  if (!aligned(q, 16) || !aligned(k_new, 16) || !aligned(v_new, 16) || !aligned(k_cache, 16) ||
      !aligned(v_cache, 16) || !aligned(out, 16))
    return layer < 0 ? fail(c, BS_ERR_INVALID_ARG, "tensor pointers must be 16-byte aligned")
                     : fail(c, BS_ERR_INVALID_ARG, "layer %d: tensor pointers must be 16-byte aligned", layer);
  return BS_OK;
}

// The bf16 attention's (request, KV head) work items, longest rows first, so
// the tail of the grid is made of short items: one workgroup per (request,
// KV head), or per (request, KV head, 32-row block) when the query group
// times the row blocks exceeds 8 waves. When one wave owns an item (G = 1,
// L <= 32), workgroup b takes the items ranked b, b + NB, b + 2 NB, ... (NB
// workgroups): every CU streams about the same number of bytes instead of
// some CUs getting only the longest rows. Allocates nothing: `items` and
// `tmp` hold attention_item_count(...) entries each.
int attention_split(int L, int Hq, int Hkv) {
  const int RB = (L + 31) / 32;
  return (Hq / Hkv) * RB > 8 ? RB : 1;
}

size_t attention_item_count(int n, int L, int Hq, int Hkv, bs_dtype dt) {
  return dt == BS_BF16 ? (size_t)n * Hkv * attention_split(L, Hq, Hkv) : 0;
}

// The single-wave kernel's list (sorted longest first): workgroup b takes
// items b, b + NB, b + 2 NB, b + 3 NB, so every workgroup holds a long and a
// short share (only when the list fills whole workgroups).
void interleave_waves(AttnItem* items, AttnItem* tmp, size_t N) {
  if (N % kMhaWaves) return;
  const size_t NB = N / kMhaWaves;
  for (size_t b = 0; b < NB; ++b)
    for (size_t j = 0; j < (size_t)kMhaWaves; ++j) tmp[b * kMhaWaves + j] = items[j * NB + b];
  std::copy(tmp, tmp + N, items);
}

void attention_items_into(AttnItem* items, AttnItem* tmp, const bs_req_desc* reqs, int n, int L, int Hq, int Hkv) {
  const int split = attention_split(L, Hq, Hkv);
  size_t N = 0;
  for (int i = 0; i < n; ++i) {
    const Geo gq = geo_of(reqs[i], L);
    for (int h = 0; h < Hkv; ++h)
      for (int rb = 0; rb < split; ++rb)
        items[N++] = AttnItem{i, h, gq.len, gq.s, gq.B, reqs[i].row, reqs[i].off, rb, 0,
                              (gq.len + kAttnTile - 1) / kAttnTile, -1, 0};
  }
  // longest first; equal lengths keep the (request, head, row block) order
  std::sort(items, items + N, [](const AttnItem& x, const AttnItem& y) {
    if (x.len != y.len) return x.len > y.len;
    if (x.req != y.req) return x.req < y.req;
    if (x.kvh != y.kvh) return x.kvh < y.kvh;
    return x.rb < y.rb;
  });
  if (Hq == Hkv && L <= 32) interleave_waves(items, tmp, N);
}

// ---- split-KV plan
// The attention kernels hold a fixed number of work slots at once: the
// shared-tile (GQA) kernel one workgroup per CU (its ring fills the LDS), the
// single-wave (MHA) kernel four waves per CU. So a launch of whole rows lasts
// at least as long as its longest row, while slots that drew short rows sit
// idle: the straggler effect of a heterogeneous batch. The plan can cut rows
// into pieces of 64-key tiles; each piece writes a partial and a merge launch
// combines a row's pieces. Its estimate of a launch, in 64-key tiles of one
// slot's loop, is the larger of
//  * the list schedule: work items longest first on the least-loaded slot
//    (what the dispatcher does with a list sorted that way), each costing
//    kPieceOverhead + its tiles, and
//  * the machine-wide bound: all items' cost over the slots, times the
//    kernel's full-load factor (a tile takes that much longer when every slot
//    runs the loop than when few do: measured 2.07 against 1.64 us on the
//    Dream-7B layer for the shared-tile kernel; the single-wave kernel streams
//    memory, about 4.8 GB/s per wave when all 1024 run and several times that
//    alone, and 2.0 picked the faster of the caps tried on an LLaDA-8B batch
//    with one 16000-token prompt: 17 tiles, 130 us, against 22 tiles, 139 us,
//    with 3.0),
// plus, when anything is cut, the merge launch. Targets T just above the
// balanced load are tried: a row longer than T - kPieceOverhead tiles is cut
// into pieces of that many tiles plus the rest. The lowest estimate wins;
// with none below the whole rows' estimate nothing is cut. So a batch that
// fills the GPU with rows of similar length runs whole, and a few long rows
// beside short ones are spread over the idle slots.
constexpr int kPlanCUs = 256;
constexpr double kPieceOverhead = 2.0;
constexpr double kMergeFixed = 3.0;        // the merge launch, in tiles
constexpr double kMergePerPart = 0.02;     // per partial read back

struct PlanShape {
  int group;          // work items per workgroup (one workgroup per CU)
  double full_load;   // per-tile slowdown with every slot busy
};

bool shared_tile_path(int L, int Hq, int Hkv) { return !(Hq == Hkv && L <= 32); }

PlanShape plan_shape(int L, int Hq, int Hkv) {
  return shared_tile_path(L, Hq, Hkv) ? PlanShape{1, 1.3} : PlanShape{kMhaWaves, 2.0};
}

int waves_per_item(int L, int Hq, int Hkv) {
  const int G = Hq / Hkv, RB = (L + 31) / 32;
  return G * (G * RB > 8 ? 1 : RB);
}

// Estimated launch time (tiles) of work items of `tiles` tiles each (sorts
// `tiles`). Items go to workgroups as the launch will place them (a group of
// ps.group items, interleaved like interleave_waves when they fill whole
// workgroups); a workgroup holds its CU until its longest item is done.
double launch_estimate(std::vector<int>& tiles, const PlanShape& ps) {
  std::sort(tiles.begin(), tiles.end(), std::greater<int>());
  const size_t N = tiles.size(), G = (size_t)ps.group;
  const size_t NB = (N + G - 1) / G;
  double total = 0.0;
  for (int t : tiles) total += kPieceOverhead + t;
  std::priority_queue<double, std::vector<double>, std::greater<double>> cu;
  for (int i = 0; i < kPlanCUs; ++i) cu.push(0.0);
  double end = 0.0;
  for (size_t b = 0; b < NB; ++b) {
    // sorted list: the workgroup's longest item is its first
    const int longest = N % G == 0 ? tiles[b] : tiles[b * G];
    const double x = cu.top() + kPieceOverhead + longest;
    cu.pop();
    cu.push(x);
    end = std::max(end, x);
  }
  return std::max(end, ps.full_load * total / ((double)kPlanCUs * G));
}

// Largest piece (tiles) of the best plan for rows of nt[i] tiles, or 0 for no cut.
int split_cap(const std::vector<int>& nt, const PlanShape& ps) {
  if (nt.empty()) return 0;
  double total = 0.0;
  for (int t : nt) total += t + kPieceOverhead;
  std::vector<int> w(nt);
  const double whole = launch_estimate(w, ps);
  const int lb = (int)std::ceil(total / ((double)kPlanCUs * ps.group));
  if (whole <= ps.full_load * lb + kMergeFixed) return 0;    // no plan can gain
  double best = whole;
  int best_cap = 0;
  for (int T = lb; T <= lb + 5; ++T) {
    const int cap = T - (int)kPieceOverhead;
    if (cap < 2) continue;
    w.clear();
    int parts = 0;
    for (int t : nt) {
      if (t <= cap) {
        w.push_back(t);
        continue;
      }
      for (int r = t; r > 0; r -= cap) w.push_back(std::min(r, cap));
      parts += (t + cap - 1) / cap;
    }
    const double est = launch_estimate(w, ps) + kMergeFixed + kMergePerPart * parts;
    if (est < best) {
      best = est;
      best_cap = cap;
    }
  }
  return best_cap;
}

// Cuts the whole rows `items` (as attention_items_into leaves them) into
// pieces of at most `cap` tiles, sorted longest first; a row's pieces take
// consecutive partial slots, and `merges` lists the rows that were cut.
// Returns the number of partial slots.
int split_items(const std::vector<AttnItem>& items, int cap, std::vector<AttnItem>& pieces,
                std::vector<AttnMerge>& merges) {
  int parts = 0;
  pieces.clear();
  merges.clear();
  for (const AttnItem& it : items) {
    const int nt = it.t1 - it.t0;
    if (cap <= 0 || nt <= cap) {
      pieces.push_back(it);
      continue;
    }
    const int np = (nt + cap - 1) / cap;
    merges.push_back(AttnMerge{it.req, it.kvh, it.rb, it.B, parts, np, 0, 0});
    for (int k = 0; k < np; ++k) {
      AttnItem p = it;
      p.t0 = k * cap;
      p.t1 = std::min(nt, (k + 1) * cap);
      p.part = parts + k;
      pieces.push_back(p);
    }
    parts += np;
  }
  std::stable_sort(pieces.begin(), pieces.end(), [](const AttnItem& x, const AttnItem& y) {
    return x.t1 - x.t0 > y.t1 - y.t0;
  });
  return parts;
}

// Partial-slot bytes of a plan with `parts` slots.
size_t part_bytes(int parts, int L, int Hq, int Hkv, int D) {
  return (size_t)parts * waves_per_item(L, Hq, Hkv) * part_wave_floats(D) * sizeof(float);
}

// Descriptors, then (bf16) the work items above, then (split) the merge list;
// meta = {descriptors, items, item count, merges, merge count, partial slots}.
void attention_blob(Blob& blob, const bs_req_desc* reqs, int n, int L, int Hq, int Hkv, bs_dtype dt, bool split) {
  blob.meta[0] = (int)blob.add(reqs, sizeof(bs_req_desc) * n);
  if (dt == BS_BF16) {
    const size_t N = attention_item_count(n, L, Hq, Hkv, dt);
    std::vector<AttnItem> items(N), tmp(N);
    attention_items_into(items.data(), tmp.data(), reqs, n, L, Hq, Hkv);
    int cap = 0;
    if (split) {
      std::vector<int> nt(N);
      for (size_t i = 0; i < N; ++i) nt[i] = items[i].t1 - items[i].t0;
      cap = split_cap(nt, plan_shape(L, Hq, Hkv));
    }
    std::vector<AttnItem> pieces;
    std::vector<AttnMerge> merges;
    const int parts = cap > 0 ? split_items(items, cap, pieces, merges) : 0;
    if (cap > 0 && !shared_tile_path(L, Hq, Hkv)) {
      std::vector<AttnItem> t2(pieces.size());
      interleave_waves(pieces.data(), t2.data(), pieces.size());
    }
    const std::vector<AttnItem>& list = cap > 0 ? pieces : items;
    blob.meta[1] = (int)blob.add(list.data(), sizeof(AttnItem) * list.size());
    blob.meta[2] = (int)list.size();
    blob.meta[3] = (int)blob.add(merges.data(), sizeof(AttnMerge) * merges.size());
    blob.meta[4] = (int)merges.size();
    blob.meta[5] = parts;
  }
}

// Launch arguments over a device blob at `dblob` laid out as `meta` says;
// `parts` holds the plan's partial slots (unused when it has none).
AttnArgs attention_args(const void* dblob, const int* meta, int L, int Hq, int Hkv, int D, int R, int W, float scale,
                        int write_back, void* parts) {
  const char* base = static_cast<const char*>(dblob);
  AttnArgs a{};
  a.reqs = reinterpret_cast<const bs_req_desc*>(base + meta[0]);
  a.items = reinterpret_cast<const AttnItem*>(base + meta[1]);
  a.n_items = meta[2];
  a.merges = reinterpret_cast<const AttnMerge*>(base + meta[3]);
  a.n_merge = meta[4];
  a.parts = static_cast<float*>(parts);
  a.L = L; a.Hq = Hq; a.Hkv = Hkv; a.D = D; a.G = Hq / Hkv; a.RB = (L + 31) / 32; a.R = R; a.W = W;
  a.RBW = a.G * a.RB > 8 ? 1 : a.RB;
  a.scale = scale > 0.0f ? scale : 1.0f / sqrtf((float)D);
  a.scale_log2e = a.scale * 1.4426950408889634f;
  a.write_back = write_back ? 1 : 0;
  return a;
}

// ---- refresh work list
// One item per (request, query head, 128-query chunk). Items that read the
// same K/V (one request and KV head) stay together on one XCD, so their tiles
// are shared through that XCD's L2: groups, heaviest first, go to the XCD with
// the least work so far, and XCD x's queue fills grid slots x, x + 8, ...
// (workgroup b runs on XCD b % 8); missing slots are empty items.
void refresh_blob(Blob& blob, const bs_req_desc* reqs, int n, int Hq, int Hkv) {
  blob.meta[0] = (int)blob.add(reqs, sizeof(bs_req_desc) * n);
  const int G = Hq / Hkv;
  struct Group {
    int64_t work;
    int i, c;
  };
  std::vector<Group> groups;
  groups.reserve((size_t)n * Hkv);
  for (int i = 0; i < n; ++i) {
    const int64_t len = (int64_t)reqs[i].p + reqs[i].g;
    for (int c = 0; c < Hkv; ++c) groups.push_back(Group{len * len * G, i, c});
  }
  std::stable_sort(groups.begin(), groups.end(), [](const Group& x, const Group& y) { return x.work > y.work; });
  constexpr int kXcd = 8;
  std::vector<RefItem> q[kXcd];
  int64_t load[kXcd] = {0, 0, 0, 0, 0, 0, 0, 0};
  for (const Group& gr : groups) {
    const int x = (int)(std::min_element(load, load + kXcd) - load);
    load[x] += gr.work;
    const bs_req_desc& r = reqs[gr.i];
    const int len = r.p + r.g;
    for (int h = gr.c * G; h < (gr.c + 1) * G; ++h)
      for (int q0 = 0; q0 < len; q0 += kRefQ) q[x].push_back(RefItem{r.row, r.off, len, h, q0, 0, 0, 0});
  }
  size_t depth = 0;
  for (int x = 0; x < kXcd; ++x) depth = std::max(depth, q[x].size());
  std::vector<RefItem> items(depth * kXcd, RefItem{-1, 0, 0, 0, 0, 0, 0, 0});
  for (int x = 0; x < kXcd; ++x)
    for (size_t k = 0; k < q[x].size(); ++k) items[x + k * kXcd] = q[x][k];
  blob.meta[1] = (int)blob.add(items.data(), sizeof(RefItem) * items.size());
  blob.meta[2] = (int)items.size();
}

// ---- decode helpers shared by the K3 entry point and the fused step
size_t decode_ws_bytes(int n, int L, int V, bs_dtype dt) {
  if (n <= 0 || L <= 0 || V <= 0 || dtype_bytes(dt) == 0) return 0;
  return dec_workspace_bytes(n, L, dec_parts(V, dtype_bytes(dt)));
}

// The fused step's workspace: the decode's, rounded up to 256 bytes, then the
// attention's partial slots (split-KV) when the caller provides room for them.
size_t step_decode_bytes(int n, int L, int V, bs_dtype dt) { return (decode_ws_bytes(n, L, V, dt) + 255) & ~size_t(255); }

// skip_ws: the caller checks (or provides) the workspace itself
int check_decode(bs_ctx* c, int n, int L, int V, bs_dtype logits_dt, int64_t logits_row_stride, float tau,
                 int q_min, const void* ws, size_t ws_bytes, bool skip_ws = false) {
  const int eb = dtype_bytes(logits_dt);
  if (!eb) return fail(c, BS_ERR_INVALID_ARG, "bad dtype %d", (int)logits_dt);
  if (L > 64) return fail(c, BS_ERR_UNSUPPORTED, "decode needs L <= 64 (L=%d)", L);
  if (V < 1) return fail(c, BS_ERR_INVALID_ARG, "V < 1");
  if ((int64_t)n * L * dec_parts(V, eb) > INT32_MAX)
    return fail(c, BS_ERR_UNSUPPORTED, "n * L * row parts exceeds the launch grid");
  if (q_min < 1) return fail(c, BS_ERR_INVALID_ARG, "q_min=%d must be >= 1", q_min);
  if (!(tau == tau)) return fail(c, BS_ERR_INVALID_ARG, "tau is NaN");
  if (logits_row_stride < V || (logits_row_stride * eb) % 16)
    return fail(c, BS_ERR_INVALID_ARG, "logits row stride %lld must be >= V and a multiple of 16 bytes",
                (long long)logits_row_stride);
  if (skip_ws) return BS_OK;
  const size_t need = decode_ws_bytes(n, L, V, logits_dt);
  if (ws_bytes < need || (need && !ws)) return fail(c, BS_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  return BS_OK;
}

int check_decode_tensors(bs_ctx* c, const void* logits, const int32_t* tokens, const uint8_t* masked,
                         const int32_t* n_unmasked, const uint8_t* done, const uint8_t* eos_seen,
                         const float* conf_out, const int32_t* pos_out, const void* ws) {
  if (!logits || !tokens || !masked || !n_unmasked || !done || !eos_seen)
    return fail(c, BS_ERR_INVALID_ARG, "tensor pointer is NULL");
  if (!aligned(logits, 16) || !aligned(tokens, 4) || !aligned(n_unmasked, 4) || !aligned(ws, 16) ||
      (conf_out && !aligned(conf_out, 4)) || (pos_out && !aligned(pos_out, 4)))
    return fail(c, BS_ERR_INVALID_ARG, "misaligned pointer (logits and ws need 16 bytes)");
  return BS_OK;
}

DecArgs decode_args(const bs_req_desc* dreqs, int n, int L, int V, bs_dtype logits_dt, const void* logits,
                    int64_t logits_row_stride, float tau, int q_min, int eos_id, int32_t* n_unmasked,
                    uint8_t* done, uint8_t* eos_seen, float* conf_out, void* ws) {
  DecArgs a{};
  a.reqs = dreqs;
  a.n = n; a.L = L; a.V = V;
  a.logits = logits; a.row_stride = logits_row_stride;
  a.tau = tau; a.q_min = q_min; a.eos_id = eos_id;
  a.n_unmasked = n_unmasked; a.done = done; a.eos_seen = eos_seen; a.conf_out = conf_out;
  a.parts = dec_parts(V, dtype_bytes(logits_dt));
  a.part = static_cast<DecPartial*>(ws);
  return a;
}

// ---- K4 segment rules (host only)
// Every segment has len >= 0, a known source kind, and source and destination
// ranges inside their boxes. Segments of length 0 copy nothing and take no
// part in the overlap rules. Destination ranges are pairwise disjoint (a
// sweep over each row in column order, keeping the furthest end seen so far,
// so no pair can hide behind another). When a source box is the destination
// box (src_alias / stg_alias), no source range of that kind meets any
// destination range.
int check_segments(bs_ctx* c, const bs_copy_seg* segs, int nseg, int R_src, int W_src, int R_stg, int W_stg,
                   int R_dst, int W_dst, bool src_alias, bool stg_alias) {
  if (nseg < 0) return fail(c, BS_ERR_INVALID_ARG, "nseg < 0");
  if (nseg > 0 && !segs) return fail(c, BS_ERR_INVALID_ARG, "segs is NULL");
  for (int i = 0; i < nseg; ++i) {
    const bs_copy_seg& g = segs[i];
    if (g.len < 0) return fail(c, BS_ERR_INVALID_ARG, "segment %d: len < 0", i);
    if (g.src_kind != 0 && g.src_kind != 1) return fail(c, BS_ERR_INVALID_ARG, "segment %d: src_kind %d", i, g.src_kind);
    const int Rs = g.src_kind ? R_stg : R_src, Ws = g.src_kind ? W_stg : W_src;
    if (g.src_row < 0 || g.src_row >= Rs || g.src_col < 0 || (int64_t)g.src_col + g.len > Ws)
      return fail(c, BS_ERR_INVALID_ARG, "segment %d: source range outside its box", i);
    if (g.dst_row < 0 || g.dst_row >= R_dst || g.dst_col < 0 || (int64_t)g.dst_col + g.len > W_dst)
      return fail(c, BS_ERR_INVALID_ARG, "segment %d: destination range outside the box", i);
  }
  std::vector<int> order;
  order.reserve((size_t)nseg);
  for (int i = 0; i < nseg; ++i)
    if (segs[i].len > 0) order.push_back(i);
  std::sort(order.begin(), order.end(), [&](int x, int y) {
    return segs[x].dst_row != segs[y].dst_row ? segs[x].dst_row < segs[y].dst_row : segs[x].dst_col < segs[y].dst_col;
  });
  int64_t reach = 0;   // furthest destination end so far in the current row
  int reach_seg = -1;
  for (size_t t = 0; t < order.size(); ++t) {
    const bs_copy_seg& y = segs[order[t]];
    if (t == 0 || segs[order[t - 1]].dst_row != y.dst_row) {
      reach = 0;
      reach_seg = -1;
    }
    if (reach_seg >= 0 && reach > y.dst_col)
      return fail(c, BS_ERR_OVERLAP, "segments %d and %d write overlapping destination cells", reach_seg, order[t]);
    if ((int64_t)y.dst_col + y.len > reach) {
      reach = (int64_t)y.dst_col + y.len;
      reach_seg = order[t];
    }
  }
  if (src_alias || stg_alias) {
    // destinations are now known disjoint and sorted: for a source range
    // [a, b) on row r only the last destination of row r starting before b
    // can meet it
    for (int i = 0; i < nseg; ++i) {
      const bs_copy_seg& g = segs[i];
      if (g.len == 0 || (g.src_kind == 0 && !src_alias) || (g.src_kind == 1 && !stg_alias)) continue;
      const int64_t a = g.src_col, b = (int64_t)g.src_col + g.len;
      auto it = std::lower_bound(order.begin(), order.end(), 0, [&](int x, int) {
        const bs_copy_seg& d = segs[x];
        return d.dst_row < g.src_row || (d.dst_row == g.src_row && d.dst_col < b);
      });
      if (it == order.begin()) continue;
      const int jj = *(it - 1);
      const bs_copy_seg& d = segs[jj];
      if (d.dst_row == g.src_row && (int64_t)d.dst_col + d.len > a)
        return fail(c, BS_ERR_OVERLAP, "segment %d reads cells that segment %d writes", i, jj);
    }
  }
  return BS_OK;
}

// ---- phase timing of the fused step
hipError_t prof_mark(bs_ctx* c, int phase, hipStream_t s) {
  Prof& p = c->prof;
  if (!p.on || p.used >= p.cap) return hipSuccess;
  return hipEventRecord(p.ev[(size_t)p.used * (kProfPhases + 1) + phase], s);
}

// Set-up of the allocation-free step for context c, on its device: the
// device address of `scratch` (resolved once per device and kept), the
// context's pinned stages and their events, and the interleave temporary.
std::mutex g_scratch_mu;
void* g_scratch_addr[64] = {};

int static_setup(bs_ctx* c) {
  if (c->device >= 64) return fail(nullptr, BS_ERR_UNSUPPORTED, "device %d: the library serves devices 0..63", c->device);
  DeviceGuard dg(c->device);
  if (!dg.ok) return fail(nullptr, BS_ERR_HIP, "hipSetDevice(%d) failed", c->device);
  {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_addr[c->device]) {
      void* p = nullptr;
      hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !p) return hip_fail(nullptr, e != hipSuccess ? e : hipErrorInvalidSymbol,
                                                 "hipGetSymbolAddress(scratch)");
      g_scratch_addr[c->device] = p;
    }
    c->stat.scratch = g_scratch_addr[c->device];
  }
  for (int k = 0; k < kStaticStages; ++k) {
    hipError_t e = hipHostMalloc(&c->stat.stage[k], kStaticBlobBytes, hipHostMallocDefault);
    if (e != hipSuccess) return hip_fail(nullptr, e, "hipHostMalloc(no-alloc stage)");
    e = hipEventCreateWithFlags(&c->stat.copied[k], hipEventDisableTiming);
    if (e != hipSuccess) return hip_fail(nullptr, e, "hipEventCreate(no-alloc stage)");
  }
  c->stat.tmp.reset(new AttnItem[kStaticBlobBytes / sizeof(AttnItem)]);
  return BS_OK;
}

}  // namespace

extern "C" {

int bs_create(bs_ctx** out, int device) {
  if (!out) return fail(nullptr, BS_ERR_INVALID_ARG, "out is NULL");
  *out = nullptr;
  int count = 0;
  hipError_t e = hipGetDeviceCount(&count);
  if (e != hipSuccess) return hip_fail(nullptr, e, "hipGetDeviceCount");
  if (device < 0 || device >= count) return fail(nullptr, BS_ERR_INVALID_ARG, "device %d of %d", device, count);
  bs_ctx* c = new bs_ctx();
  c->device = device;
  int st = static_setup(c);
  if (st) {
    bs_destroy(c);
    return st;
  }
  *out = c;
  return BS_OK;
}

int bs_destroy(bs_ctx* c) {
  if (!c) return BS_OK;
  DeviceGuard dg(c->device);
  for (hipEvent_t e : c->prof.ev) (void)hipEventDestroy(e);
  for (int k = 0; k < kStaticStages; ++k) {
    if (c->stat.copied[k]) {
      (void)hipEventSynchronize(c->stat.copied[k]);
      (void)hipEventDestroy(c->stat.copied[k]);
    }
    if (c->stat.stage[k]) (void)hipHostFree(c->stat.stage[k]);
  }
  for (auto& p : c->slots) {
    Slot& sl = *p;
    if (sl.live) (void)hipEventSynchronize(sl.done);
    if (sl.d) (void)hipFree(sl.d);
    if (sl.h) (void)hipHostFree(sl.h);
    if (sl.ready) (void)hipEventDestroy(sl.ready);
    if (sl.done) (void)hipEventDestroy(sl.done);
  }
  delete c;
  return BS_OK;
}

const char* bs_status_string(int st) {
  switch (st) {
    case BS_OK: return "BS_OK";
    case BS_ERR_INVALID_ARG: return "BS_ERR_INVALID_ARG";
    case BS_ERR_UNSUPPORTED: return "BS_ERR_UNSUPPORTED";
    case BS_ERR_DESCRIPTOR: return "BS_ERR_DESCRIPTOR";
    case BS_ERR_OVERLAP: return "BS_ERR_OVERLAP";
    case BS_ERR_WORKSPACE: return "BS_ERR_WORKSPACE";
    case BS_ERR_HIP: return "BS_ERR_HIP";
    default: return "BS_UNKNOWN_STATUS";
  }
}

const char* bs_last_error(const bs_ctx* c) { return c ? c->err.c_str() : g_err.c_str(); }

int bs_validate_requests(const bs_req_desc* reqs, int n, int L, int R, int W) {
  return check_reqs(nullptr, reqs, n, L, R, W);
}

int bs_validate_segments(const bs_copy_seg* segs, int nseg, int R_src, int W_src, int R_stg, int W_stg, int R_dst,
                         int W_dst, int src_is_dst, int stg_is_dst) {
  return check_segments(nullptr, segs, nseg, R_src, W_src, R_stg, W_stg, R_dst, W_dst, src_is_dst != 0,
                        stg_is_dst != 0);
}

// ------------------------------------------------------------------ K1
static int gather_common(bs_ctx* c, const bs_req_desc* reqs, int n, int L, int R, int W, int nt,
                         const void* const* dense, const int64_t* stride, const int* eb, void* const* compact,
                         bool gather, int32_t* pos, void* stream) {
  if (!c) return fail(nullptr, BS_ERR_INVALID_ARG, "ctx is NULL");
  int st = check_reqs(c, reqs, n, L, R, W);
  if (st) return st;
  if (nt < 1 || nt > kMaxGather) return fail(c, BS_ERR_INVALID_ARG, "ntensors=%d outside [1, %d]", nt, kMaxGather);
  if (!dense || !stride || !eb || !compact) return fail(c, BS_ERR_INVALID_ARG, "tensor array is NULL");
  GatherSet g{};
  g.count = nt;
  for (int k = 0; k < nt; ++k) {
    const int e = eb[k];
    if (!(e == 1 || e == 2 || e == 4 || e == 8 || e == 16))
      return fail(c, BS_ERR_UNSUPPORTED, "tensor %d: elem_bytes=%d (supported: 1, 2, 4, 8, 16)", k, e);
    if (n == 0) continue;
    if (!dense[k] || !compact[k]) return fail(c, BS_ERR_INVALID_ARG, "tensor %d: pointer is NULL", k);
    if (stride[k] < (int64_t)W * e)
      return fail(c, BS_ERR_INVALID_ARG, "tensor %d: row stride %lld < W*elem", k, (long long)stride[k]);
    if (stride[k] % e || !aligned(dense[k], e) || !aligned(compact[k], e))
      return fail(c, BS_ERR_INVALID_ARG, "tensor %d: pointers and row stride must be multiples of elem_bytes", k);
    g.dense[k] = dense[k];
    g.compact[k] = compact[k];
    g.stride[k] = stride[k];
    g.eb[k] = e;
  }
  if (pos && !aligned(pos, 4)) return fail(c, BS_ERR_INVALID_ARG, "pos_out must be 4-byte aligned");
  if (n == 0) return BS_OK;
  DeviceGuard dg(c->device);
  if (!dg.ok) return fail(c, BS_ERR_HIP, "hipSetDevice(%d) failed", c->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  Slot* sl = nullptr;
  st = upload_reqs(c, s, reqs, n, &sl);
  if (st) return st;
  const bs_req_desc* dreqs = static_cast<const bs_req_desc*>(sl->d);
  hipError_t e = gather ? launch_gather(dreqs, n, L, g, pos, s) : launch_scatter(dreqs, n, L, g, s);
  return finish(c, sl, s, e, gather ? "gather launch" : "scatter launch");
}

int bs_gather_active_blocks(bs_ctx* c, const bs_req_desc* reqs, int n, int L, int R, int W,
                            const void* src, int64_t src_row_stride_bytes, int elem_bytes,
                            void* dst, int32_t* pos_out, void* stream) {
  return gather_common(c, reqs, n, L, R, W, 1, &src, &src_row_stride_bytes, &elem_bytes, &dst, true, pos_out, stream);
}

int bs_scatter_active_blocks(bs_ctx* c, const bs_req_desc* reqs, int n, int L, int R, int W,
                             const void* src_compact, int elem_bytes, void* dst_dense,
                             int64_t dst_row_stride_bytes, void* stream) {
  const void* dense = dst_dense;
  void* compact = const_cast<void*>(src_compact);
  return gather_common(c, reqs, n, L, R, W, 1, &dense, &dst_row_stride_bytes, &elem_bytes, &compact, false,
                       nullptr, stream);
}

int bs_gather_active_blocks_n(bs_ctx* c, const bs_req_desc* reqs, int n, int L, int R, int W, int ntensors,
                              const void* const* src, const int64_t* src_row_stride_bytes,
                              const int* elem_bytes, void* const* dst, int32_t* pos_out, void* stream) {
  return gather_common(c, reqs, n, L, R, W, ntensors, src, src_row_stride_bytes, elem_bytes, dst, true, pos_out,
                       stream);
}

int bs_scatter_active_blocks_n(bs_ctx* c, const bs_req_desc* reqs, int n, int L, int R, int W, int ntensors,
                               const void* const* src_compact, const int* elem_bytes, void* const* dst_dense,
                               const int64_t* dst_row_stride_bytes, void* stream) {
  // the kernel writes through the dense pointers; the set stores them as const
  return gather_common(c, reqs, n, L, R, W, ntensors, const_cast<const void* const*>(dst_dense),
                       dst_row_stride_bytes, elem_bytes, const_cast<void* const*>(src_compact), false, nullptr,
                       stream);
}

// ------------------------------------------------------------------ K2
size_t bs_attention_workspace_bytes(const bs_req_desc* reqs, int n, int L, int Hq, int Hkv, int D,
                                    bs_dtype dt) {
  if (!reqs || n <= 0 || dt != BS_BF16 || L < 1 || L > 64 || Hkv < 1 || Hq < Hkv || Hq % Hkv || (D != 64 && D != 128))
    return 0;
  const size_t N = attention_item_count(n, L, Hq, Hkv, dt);
  std::vector<AttnItem> items(N), tmp(N);
  attention_items_into(items.data(), tmp.data(), reqs, n, L, Hq, Hkv);
  std::vector<int> nt(N);
  for (size_t i = 0; i < N; ++i) nt[i] = std::max(items[i].t1 - items[i].t0, 0);
  const int cap = split_cap(nt, plan_shape(L, Hq, Hkv));
  int parts = 0;
  if (cap > 0)
    for (int t : nt)
      if (t > cap) parts += (t + cap - 1) / cap;
  return part_bytes(parts, L, Hq, Hkv, D);
}

int bs_attention_work_list(const bs_req_desc* reqs, int n, int L, int Hq, int Hkv, int D, bs_dtype dt, int split,
                           int32_t* items, int max_items, int* n_items, int* n_parts) {
  if (!n_items || !n_parts || (max_items > 0 && !items) || n < 0 || (n > 0 && !reqs))
    return fail(nullptr, BS_ERR_INVALID_ARG, "bad work-list arguments");
  if (dt != BS_BF16 || L < 1 || L > 64 || Hkv < 1 || Hq < Hkv || Hq % Hkv || (D != 64 && D != 128))
    return fail(nullptr, BS_ERR_UNSUPPORTED, "work lists exist for the bf16 kernels only");
  Blob blob;
  attention_blob(blob, reqs, n, L, Hq, Hkv, dt, split != 0);
  const int N = blob.meta[2];
  *n_items = N;
  *n_parts = blob.meta[5];
  const AttnItem* it = reinterpret_cast<const AttnItem*>(blob.bytes.data() + blob.meta[1]);
  for (int i = 0; i < std::min(N, max_items); ++i) {
    const int32_t v[6] = {it[i].req, it[i].kvh, it[i].rb, it[i].t0, it[i].t1, it[i].part};
    std::memcpy(items + 6 * (size_t)i, v, sizeof v);
  }
  return BS_OK;
}

// The attention blob of a call: split (split-KV) when `room` bytes of partial
// slots hold the plan's, else every row whole.
int attention_upload(bs_ctx* c, hipStream_t s, const bs_req_desc* reqs, int n, int L, int Hq, int Hkv, int D,
                     bs_dtype dt, size_t room, Slot** out) {
  for (int split = room > 0 ? 1 : 0; split >= 0; --split) {
    int st = upload(c, s, Key('A', {n, L, Hq, Hkv, (int64_t)dt, split}, reqs, sizeof(bs_req_desc) * n),
                    [&](Blob& blob) { attention_blob(blob, reqs, n, L, Hq, Hkv, dt, split != 0); }, out);
    if (st) return st;
    if (part_bytes((*out)->meta[5], L, Hq, Hkv, D) <= room) return BS_OK;
  }
  return BS_OK;   // not reached: the whole-row blob has no partial slots
}

int bs_dual_cache_block_attention(bs_ctx* c, const bs_req_desc* reqs, int n, int L, int Hq,
                                  int Hkv, int D, bs_dtype dt, float scale, const void* q,
                                  const void* k_new, const void* v_new, void* k_cache,
                                  void* v_cache, int R, int W, int write_back, void* out,
                                  void* ws, size_t ws_bytes, void* stream) {
  if (!c) return fail(nullptr, BS_ERR_INVALID_ARG, "ctx is NULL");
  int st = check_reqs(c, reqs, n, L, R, W);
  if (st) return st;
  st = check_attention(c, n, L, Hq, Hkv, D, dt);
  if (st) return st;
  if (n == 0) return BS_OK;
  st = check_attention_tensors(c, q, k_new, v_new, k_cache, v_cache, out, -1);
  if (st) return st;
  DeviceGuard dg(c->device);
  if (!dg.ok) return fail(c, BS_ERR_HIP, "hipSetDevice(%d) failed", c->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  Slot* sl = nullptr;
  st = attention_upload(c, s, reqs, n, L, Hq, Hkv, D, dt, ws ? ws_bytes : 0, &sl);
  if (st) return st;
  AttnArgs a = attention_args(sl->d, sl->meta, L, Hq, Hkv, D, R, W, scale, write_back, ws);
  a.q = q; a.k_new = k_new; a.v_new = v_new; a.k_cache = k_cache; a.v_cache = v_cache; a.out = out;
  hipError_t e = dt == BS_F32 ? launch_attn_f32(a, n, s) : launch_attn_bf16(a, s);
  return finish(c, sl, s, e, "attention launch");
}

// ------------------------------------------------------------------ K3
size_t bs_decode_workspace_bytes(int n, int L, int V, bs_dtype dt) { return decode_ws_bytes(n, L, V, dt); }

size_t bs_step_workspace_bytes(const bs_req_desc* reqs, int n, int L, int Hq, int Hkv, int D, bs_dtype dt, int V,
                               bs_dtype logits_dt) {
  return step_decode_bytes(n, L, V, logits_dt) + bs_attention_workspace_bytes(reqs, n, L, Hq, Hkv, D, dt);
}

int bs_parallel_decode(bs_ctx* c, const bs_req_desc* reqs, int n, int L, int V,
                       bs_dtype logits_dt, const void* logits, int64_t logits_row_stride,
                       int32_t* tokens, uint8_t* masked, float tau, int32_t q_min, int32_t eos_id,
                       int32_t* n_unmasked, uint8_t* done, uint8_t* eos_seen, float* conf_out,
                       void* ws, size_t ws_bytes, void* stream) {
  if (!c) return fail(nullptr, BS_ERR_INVALID_ARG, "ctx is NULL");
  if (n < 0) return fail(c, BS_ERR_INVALID_ARG, "n < 0");
  if (n > 0 && !reqs) return fail(c, BS_ERR_INVALID_ARG, "reqs is NULL");
  if (L < 1) return fail(c, BS_ERR_DESCRIPTOR, "L < 1");
  for (int i = 0; i < n; ++i) {
    const bs_req_desc& r = reqs[i];
    const int64_t K = ((int64_t)r.g + L - 1) / L;
    if (r.p < 0 || r.g < 1 || r.k < 0 || r.k >= K)
      return fail(c, BS_ERR_DESCRIPTOR, "request %d: p=%d g=%d k=%d invalid for L=%d", i, r.p, r.g, r.k, L);
  }
  int st = check_decode(c, n, L, V, logits_dt, logits_row_stride, tau, q_min, ws, ws_bytes);
  if (st) return st;
  if (n == 0) return BS_OK;
  st = check_decode_tensors(c, logits, tokens, masked, n_unmasked, done, eos_seen, conf_out, nullptr, ws);
  if (st) return st;
  DeviceGuard dg(c->device);
  if (!dg.ok) return fail(c, BS_ERR_HIP, "hipSetDevice(%d) failed", c->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  Slot* sl = nullptr;
  st = upload_reqs(c, s, reqs, n, &sl);
  if (st) return st;
  DecArgs a = decode_args(static_cast<const bs_req_desc*>(sl->d), n, L, V, logits_dt, logits, logits_row_stride,
                          tau, q_min, eos_id, n_unmasked, done, eos_seen, conf_out, ws);
  a.tokens = tokens; a.masked = masked;
  hipError_t e = launch_decode(a, logits_dt, s);
  return finish(c, sl, s, e, "decode launch");
}

// ------------------------------------------------------------------ K3 with the output head
size_t bs_lm_head_workspace_bytes(int n, int L, int V) {
  if (n <= 0 || L <= 0 || V <= 0) return 0;
  return lm_workspace_bytes(n, L, V);
}

size_t bs_lm_head_pack_bytes(int V, int d) {
  if (V <= 0 || d <= 0) return 0;
  return lm_packed_bytes(V, d);
}

int bs_lm_head_pack(bs_ctx* c, const void* w_vocab, int64_t w_row_stride, int V, int d, bs_dtype dt,
                    void* w_packed, size_t packed_bytes, void* stream) {
  if (!c) return fail(nullptr, BS_ERR_INVALID_ARG, "ctx is NULL");
  if (dt != BS_BF16) return fail(c, BS_ERR_UNSUPPORTED, "the output head runs in bf16 only (dt=%d)", (int)dt);
  if (V < 1) return fail(c, BS_ERR_INVALID_ARG, "V < 1");
  if (d < kLmKT || d % kLmKT) return fail(c, BS_ERR_UNSUPPORTED, "d=%d must be a positive multiple of %d", d, kLmKT);
  if (w_row_stride < d || w_row_stride % 8)
    return fail(c, BS_ERR_INVALID_ARG, "w_row_stride %lld must be >= d and a multiple of 8",
                (long long)w_row_stride);
  if (packed_bytes < lm_packed_bytes(V, d))
    return fail(c, BS_ERR_WORKSPACE, "packed buffer %zu < %zu bytes", packed_bytes, lm_packed_bytes(V, d));
  if (!w_vocab || !w_packed) return fail(c, BS_ERR_INVALID_ARG, "tensor pointer is NULL");
  if (!aligned(w_vocab, 16) || !aligned(w_packed, 16)) return fail(c, BS_ERR_INVALID_ARG, "misaligned pointer");
  DeviceGuard dg(c->device);
  if (!dg.ok) return fail(c, BS_ERR_HIP, "hipSetDevice(%d) failed", c->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  hipError_t e = launch_lm_pack(static_cast<const uint16_t*>(w_vocab), w_row_stride, V, d,
                                static_cast<uint16_t*>(w_packed), s);
  if (e != hipSuccess) return hip_fail(c, e, "output-head pack launch");
  return BS_OK;
}

int bs_lm_head_decode(bs_ctx* c, const bs_req_desc* reqs, int n, int L, int d, int V, bs_dtype dt,
                      const void* hidden, const void* w_packed, int32_t* tokens, uint8_t* masked, float tau,
                      int32_t q_min, int32_t eos_id, int32_t* n_unmasked, uint8_t* done, uint8_t* eos_seen,
                      float* conf_out, void* ws, size_t ws_bytes, void* stream) {
  if (!c) return fail(nullptr, BS_ERR_INVALID_ARG, "ctx is NULL");
  if (n < 0) return fail(c, BS_ERR_INVALID_ARG, "n < 0");
  if (n > 0 && !reqs) return fail(c, BS_ERR_INVALID_ARG, "reqs is NULL");
  if (L < 1) return fail(c, BS_ERR_DESCRIPTOR, "L < 1");
  for (int i = 0; i < n; ++i) {
    const bs_req_desc& r = reqs[i];
    const int64_t K = ((int64_t)r.g + L - 1) / L;
    if (r.p < 0 || r.g < 1 || r.k < 0 || r.k >= K)
      return fail(c, BS_ERR_DESCRIPTOR, "request %d: p=%d g=%d k=%d invalid for L=%d", i, r.p, r.g, r.k, L);
  }
  if (dt != BS_BF16) return fail(c, BS_ERR_UNSUPPORTED, "the output head runs in bf16 only (dt=%d)", (int)dt);
  if (L > 64) return fail(c, BS_ERR_UNSUPPORTED, "decode needs L <= 64 (L=%d)", L);
  if (d < kLmKT || d % kLmKT) return fail(c, BS_ERR_UNSUPPORTED, "d=%d must be a positive multiple of %d", d, kLmKT);
  if (V < 1) return fail(c, BS_ERR_INVALID_ARG, "V < 1");
  if ((int64_t)n * L > 65536) return fail(c, BS_ERR_UNSUPPORTED, "n * L = %lld exceeds 65536", (long long)n * L);
  if (q_min < 1) return fail(c, BS_ERR_INVALID_ARG, "q_min=%d must be >= 1", q_min);
  if (!(tau == tau)) return fail(c, BS_ERR_INVALID_ARG, "tau is NaN");
  const size_t need = bs_lm_head_workspace_bytes(n, L, V);
  if (ws_bytes < need || (need && !ws)) return fail(c, BS_ERR_WORKSPACE, "workspace %zu < %zu bytes", ws_bytes, need);
  if (n == 0) return BS_OK;
  if (!hidden || !w_packed || !tokens || !masked || !n_unmasked || !done || !eos_seen)
    return fail(c, BS_ERR_INVALID_ARG, "tensor pointer is NULL");
  if (!aligned(hidden, 16) || !aligned(w_packed, 16) || !aligned(tokens, 4) || !aligned(n_unmasked, 4) ||
      !aligned(ws, 16) || (conf_out && !aligned(conf_out, 4)))
    return fail(c, BS_ERR_INVALID_ARG, "misaligned pointer (hidden, w_packed and ws need 16 bytes)");
  DeviceGuard dg(c->device);
  if (!dg.ok) return fail(c, BS_ERR_HIP, "hipSetDevice(%d) failed", c->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  Slot* sl = nullptr;
  int st = upload_reqs(c, s, reqs, n, &sl);
  if (st) return st;
  const bs_req_desc* dreqs = static_cast<const bs_req_desc*>(sl->d);
  char* wsb = static_cast<char*>(ws);
  LmArgs m{};
  m.reqs = dreqs;
  m.n = n; m.L = L; m.d = d; m.V = V;
  m.hidden = static_cast<const uint16_t*>(hidden);
  m.w = static_cast<const uint16_t*>(w_packed);
  m.masked = masked;
  m.count = reinterpret_cast<int32_t*>(wsb);
  m.rows = reinterpret_cast<int32_t*>(wsb + 16);
  m.row_part = reinterpret_cast<DecPartial*>(wsb + 16 + lm_rows_bytes(n, L));
  m.slices = m.row_part + (size_t)n * L;
  m.parts = lm_parts(V);
  DecArgs a = decode_args(dreqs, n, L, V, BS_F32, nullptr, V, tau, q_min, eos_id, n_unmasked, done, eos_seen,
                          conf_out, m.row_part);
  a.parts = 1;
  a.tokens = tokens; a.masked = masked;
  // phase events (when the ring is armed): row list | GEMM | merge + selection
  hipError_t e = prof_mark(c, 0, s);
  if (e == hipSuccess) e = launch_lm_rows(m, s);
  if (e == hipSuccess) e = prof_mark(c, 1, s);
  if (e == hipSuccess) e = launch_lm_gemm(m, s);
  if (e == hipSuccess) e = prof_mark(c, 2, s);
  if (e == hipSuccess) e = launch_lm_merge(m, s);
  if (e == hipSuccess) e = launch_decode_select(a, s);
  if (e == hipSuccess) e = prof_mark(c, 3, s);
  if (e == hipSuccess && c->prof.on && c->prof.used < c->prof.cap) ++c->prof.used;
  return finish(c, sl, s, e, "output-head decode launch");
}

// ------------------------------------------------------------------ dual-cache refresh
int bs_dual_cache_refresh(bs_ctx* c, const bs_req_desc* reqs, int n, int L, int Hq, int Hkv, int D, bs_dtype dt,
                          float scale, float rope_base, const void* q, const void* k, const void* v, int R, int W,
                          void* k_cache, void* v_cache, void* out, void* stream) {
  if (!c) return fail(nullptr, BS_ERR_INVALID_ARG, "ctx is NULL");
  int st = check_reqs(c, reqs, n, L, R, W);
  if (st) return st;
  if (dt != BS_BF16) return fail(c, BS_ERR_UNSUPPORTED, "the refresh runs in bf16 only (dt=%d)", (int)dt);
  if (Hq < 1 || Hkv < 1) return fail(c, BS_ERR_INVALID_ARG, "Hq, Hkv must be >= 1");
  if (Hq % Hkv) return fail(c, BS_ERR_UNSUPPORTED, "Hq=%d not a multiple of Hkv=%d", Hq, Hkv);
  if (D != 128) return fail(c, BS_ERR_UNSUPPORTED, "the refresh needs D = 128 (D=%d)", D);
  if (!(rope_base == rope_base)) return fail(c, BS_ERR_INVALID_ARG, "rope_base is NaN");
  if ((int64_t)R * W * Hq > INT32_MAX) return fail(c, BS_ERR_UNSUPPORTED, "R * W * Hq exceeds 2^31");
  if (n > 65535) return fail(c, BS_ERR_UNSUPPORTED, "n=%d requests exceed the 65535 of one launch", n);
  if (n == 0) return BS_OK;
  if (!q || !k || !v || !k_cache || !v_cache || !out) return fail(c, BS_ERR_INVALID_ARG, "tensor pointer is NULL");
  if (!aligned(q, 16) || !aligned(k, 16) || !aligned(v, 16) || !aligned(k_cache, 16) || !aligned(v_cache, 16) ||
      !aligned(out, 16))
    return fail(c, BS_ERR_INVALID_ARG, "tensor pointers must be 16-byte aligned");
  DeviceGuard dg(c->device);
  if (!dg.ok) return fail(c, BS_ERR_HIP, "hipSetDevice(%d) failed", c->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  Slot* sl = nullptr;
  st = upload(c, s, Key('F', {n, Hq, Hkv}, reqs, sizeof(bs_req_desc) * n),
              [&](Blob& blob) { refresh_blob(blob, reqs, n, Hq, Hkv); }, &sl);
  if (st) return st;
  int max_len = 0;
  for (int i = 0; i < n; ++i) max_len = std::max(max_len, reqs[i].p + reqs[i].g);
  const char* base = static_cast<const char*>(sl->d);
  const bool rope = rope_base > 0.0f;
  const float nl2b = rope ? (float)(-2.0 * std::log2((double)rope_base) / D) : 0.0f;
  RefKvArgs kv{};
  kv.reqs = reinterpret_cast<const bs_req_desc*>(base + sl->meta[0]);
  kv.Hkv = Hkv; kv.W = W; kv.nl2b = nl2b; kv.rope = rope ? 1 : 0;
  kv.k = static_cast<const uint16_t*>(k); kv.v = static_cast<const uint16_t*>(v);
  kv.k_cache = static_cast<uint16_t*>(k_cache); kv.v_cache = static_cast<uint16_t*>(v_cache);
  RefArgs a{};
  a.items = reinterpret_cast<const RefItem*>(base + sl->meta[1]);
  a.Hq = Hq; a.Hkv = Hkv; a.G = Hq / Hkv; a.W = W;
  const float sc = scale > 0.0f ? scale : 1.0f / sqrtf((float)D);
  a.scale_log2e = sc * 1.4426950408889634f;
  a.nl2b = nl2b; a.rope = kv.rope;
  a.q = static_cast<const uint16_t*>(q); a.out = static_cast<uint16_t*>(out);
  a.k_cache = kv.k_cache; a.v_cache = kv.v_cache;
  // phase events (when the ring is armed): rotated keys and values | attention
  hipError_t e = prof_mark(c, 0, s);
  if (e == hipSuccess) e = launch_refresh_kv(kv, n, max_len, s);
  if (e == hipSuccess) e = prof_mark(c, 1, s);
  if (e == hipSuccess) e = launch_refresh_attn(a, sl->meta[2], s);
  if (e == hipSuccess) e = prof_mark(c, 2, s);
  if (e == hipSuccess) e = prof_mark(c, 3, s);
  if (e == hipSuccess && c->prof.on && c->prof.used < c->prof.cap) ++c->prof.used;
  return finish(c, sl, s, e, "refresh launch");
}

// ------------------------------------------------------------------ fused step
// Checks shared by bs_mixed_state_step and its allocation-free variant (the
// decode workspace is checked by the caller).
static int check_step(bs_ctx* c, const bs_req_desc* reqs, int n, int L, int R, int W, int n_layers, int Hq, int Hkv,
                      int D, bs_dtype dt, const void* const* q, const void* const* k_new, const void* const* v_new,
                      void* const* k_cache, void* const* v_cache, void* const* out, int V, bs_dtype logits_dt,
                      int64_t logits_row_stride, int64_t tokens_row_stride, int64_t masked_row_stride, float tau,
                      int32_t q_min) {
  if (!c) return fail(nullptr, BS_ERR_INVALID_ARG, "ctx is NULL");
  int st = check_reqs(c, reqs, n, L, R, W);
  if (st) return st;
  if (n_layers < 0) return fail(c, BS_ERR_INVALID_ARG, "n_layers < 0");
  if (n_layers > 0) {
    st = check_attention(c, n, L, Hq, Hkv, D, dt);
    if (st) return st;
  }
  // the workspace is checked separately: pass a size that always suffices
  st = check_decode(c, n, L, V, logits_dt, logits_row_stride, tau, q_min, nullptr, 0, true);
  if (st) return st;
  if (tokens_row_stride < W || masked_row_stride < W)
    return fail(c, BS_ERR_INVALID_ARG, "token/mask row strides must be >= W");
  if (n == 0) return BS_OK;
  if (n_layers > 0 && (!q || !k_new || !v_new || !k_cache || !v_cache || !out))
    return fail(c, BS_ERR_INVALID_ARG, "layer pointer array is NULL");
  for (int l = 0; l < n_layers; ++l) {
    st = check_attention_tensors(c, q[l], k_new[l], v_new[l], k_cache[l], v_cache[l], out[l], l);
    if (st) return st;
  }
  return BS_OK;
}

// Enqueues the step over the device blob `dblob` (descriptors and attention
// work items, laid out as `meta` says) with decode partials in `ws`.
static hipError_t step_launch(bs_ctx* c, const void* dblob, const int* meta, int n, int L, int R, int W, int n_layers,
                              int Hq, int Hkv, int D, bs_dtype dt, float scale, int write_back, const void* const* q,
                              const void* const* k_new, const void* const* v_new, void* const* k_cache,
                              void* const* v_cache, void* const* out, int V, bs_dtype logits_dt, const void* logits,
                              int64_t logits_row_stride, int32_t* tokens, int64_t tokens_row_stride, uint8_t* masked,
                              int64_t masked_row_stride, float tau, int32_t q_min, int32_t eos_id,
                              int32_t* n_unmasked, uint8_t* done, uint8_t* eos_seen, float* conf_out,
                              int32_t* pos_out, void* ws, void* part_slots, hipStream_t s) {
  hipError_t e = prof_mark(c, 0, s);
  AttnArgs a = attention_args(dblob, meta, L, Hq, Hkv, D, R, W, scale, write_back, part_slots);
  // the bf16 attention of the first layer also leaves each request's block
  // mask word behind the decode partials, for the row reductions below
  const int parts = dec_parts(V, dtype_bytes(logits_dt));
  uint64_t* words = reinterpret_cast<uint64_t*>(static_cast<unsigned char*>(ws) + dec_parts_bytes(n, L, parts));
  const bool use_words = n_layers > 0 && dt == BS_BF16;
  for (int l = 0; l < n_layers && e == hipSuccess; ++l) {
    a.q = q[l]; a.k_new = k_new[l]; a.v_new = v_new[l]; a.k_cache = k_cache[l]; a.v_cache = v_cache[l]; a.out = out[l];
    a.mask_words = use_words && l == 0 ? words : nullptr;
    a.masked = masked; a.msk_rs = masked_row_stride;
    e = dt == BS_F32 ? launch_attn_f32(a, n, s) : launch_attn_bf16(a, s);
  }
  if (e == hipSuccess) e = prof_mark(c, 1, s);
  if (e == hipSuccess) {
    DecArgs d = decode_args(a.reqs, n, L, V, logits_dt, logits, logits_row_stride, tau, q_min, eos_id, n_unmasked,
                            done, eos_seen, conf_out, ws);
    d.tokens = tokens; d.masked = masked;
    d.dense = 1; d.tok_rs = tokens_row_stride; d.msk_rs = masked_row_stride;
    d.pos_out = pos_out;
    d.words = use_words ? words : nullptr;
    e = launch_decode_marked(d, logits_dt, s, [&](int ph) { return prof_mark(c, ph, s); });
  }
  if (e == hipSuccess && c->prof.on && c->prof.used < c->prof.cap) ++c->prof.used;
  return e;
}

int bs_mixed_state_step(bs_ctx* c, const bs_req_desc* reqs, int n, int L, int R, int W, int n_layers, int Hq,
                        int Hkv, int D, bs_dtype dt, float scale, int write_back, const void* const* q,
                        const void* const* k_new, const void* const* v_new, void* const* k_cache,
                        void* const* v_cache, void* const* out, int V, bs_dtype logits_dt, const void* logits,
                        int64_t logits_row_stride, int32_t* tokens, int64_t tokens_row_stride, uint8_t* masked,
                        int64_t masked_row_stride, float tau, int32_t q_min, int32_t eos_id, int32_t* n_unmasked,
                        uint8_t* done, uint8_t* eos_seen, float* conf_out, int32_t* pos_out, void* ws,
                        size_t ws_bytes, void* stream) {
  int st = check_step(c, reqs, n, L, R, W, n_layers, Hq, Hkv, D, dt, q, k_new, v_new, k_cache, v_cache, out, V,
                      logits_dt, logits_row_stride, tokens_row_stride, masked_row_stride, tau, q_min);
  if (st) return st;
  st = check_decode(c, n, L, V, logits_dt, logits_row_stride, tau, q_min, ws, ws_bytes, false);
  if (st) return st;
  if (n == 0) return BS_OK;
  st = check_decode_tensors(c, logits, tokens, masked, n_unmasked, done, eos_seen, conf_out, pos_out, ws);
  if (st) return st;
  DeviceGuard dg(c->device);
  if (!dg.ok) return fail(c, BS_ERR_HIP, "hipSetDevice(%d) failed", c->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  // the workspace past the decode's (rounded to 256 bytes) holds the
  // attention's partial slots when it is large enough for the split plan
  const size_t dws = step_decode_bytes(n, L, V, logits_dt);
  Slot* sl = nullptr;
  st = attention_upload(c, s, reqs, n, L, Hq, Hkv, D, dt, n_layers > 0 && ws_bytes > dws ? ws_bytes - dws : 0, &sl);
  if (st) return st;
  hipError_t e = step_launch(c, sl->d, sl->meta, n, L, R, W, n_layers, Hq, Hkv, D, dt, scale, write_back, q, k_new,
                             v_new, k_cache, v_cache, out, V, logits_dt, logits, logits_row_stride, tokens,
                             tokens_row_stride, masked, masked_row_stride, tau, q_min, eos_id, n_unmasked, done,
                             eos_seen, conf_out, pos_out, ws, static_cast<unsigned char*>(ws) + dws, s);
  return finish(c, sl, s, e, "step launch");
}

// ------------------------------------------------------------------ fused step without allocation
// The step for callers that cannot allocate: the descriptors, the attention
// work items and the decode partials live in this device's `scratch` array
// (the library's static device memory), whose address set-up resolved. The
// blob is built in one of the context's pinned stages (allocated by
// bs_create) and copied into the array on the call's stream.
int bs_mixed_state_step_noalloc(bs_ctx* c, const bs_req_desc* reqs, int n, int L, int R, int W, int n_layers,
                                int Hq, int Hkv, int D, bs_dtype dt, float scale, int write_back,
                                const void* const* q, const void* const* k_new, const void* const* v_new,
                                void* const* k_cache, void* const* v_cache, void* const* out, int V,
                                bs_dtype logits_dt, const void* logits, int64_t logits_row_stride, int32_t* tokens,
                                int64_t tokens_row_stride, uint8_t* masked, int64_t masked_row_stride, float tau,
                                int32_t q_min, int32_t eos_id, int32_t* n_unmasked, uint8_t* done,
                                uint8_t* eos_seen, float* conf_out, int32_t* pos_out, void* stream) {
  int st = check_step(c, reqs, n, L, R, W, n_layers, Hq, Hkv, D, dt, q, k_new, v_new, k_cache, v_cache, out, V,
                      logits_dt, logits_row_stride, tokens_row_stride, masked_row_stride, tau, q_min);
  if (st) return st;
  StaticPath& sp = c->stat;
  const size_t n_items = n_layers > 0 ? attention_item_count(n, L, Hq, Hkv, dt) : 0;   // no attention, no work list
  const size_t items_off = ((size_t)n * sizeof(bs_req_desc) + 15) & ~size_t(15);
  const size_t blob_bytes = items_off + n_items * sizeof(AttnItem);
  if (blob_bytes > kStaticBlobBytes)
    return fail(c, BS_ERR_UNSUPPORTED, "descriptors and work items (%zu bytes for n=%d, Hkv=%d) exceed the %zu "
                "bytes the no-alloc step reserves for them", blob_bytes, n, Hkv, kStaticBlobBytes);
  const size_t part_bytes = decode_ws_bytes(n, L, V, logits_dt);
  if (part_bytes > kStaticPartBytes)
    return fail(c, BS_ERR_UNSUPPORTED, "decode partials (%zu bytes for n=%d, L=%d, V=%d) exceed the %zu bytes "
                "the no-alloc step reserves for them", part_bytes, n, L, V, kStaticPartBytes);
  if (n == 0) return BS_OK;
  unsigned char* dscratch = static_cast<unsigned char*>(sp.scratch);
  st = check_decode_tensors(c, logits, tokens, masked, n_unmasked, done, eos_seen, conf_out, pos_out,
                            dscratch + kStaticBlobBytes);
  if (st) return st;
  DeviceGuard dg(c->device);
  if (!dg.ok) return fail(c, BS_ERR_HIP, "hipSetDevice(%d) failed", c->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  // a stage whose previous copy has completed; only when every stage is
  // still being copied from does the call wait, for the oldest
  int k = -1;
  for (int t = 0; t < kStaticStages && k < 0; ++t) {
    const int cand = (sp.next + t) % kStaticStages;
    const hipError_t q_ = hipEventQuery(sp.copied[cand]);
    if (q_ == hipSuccess) k = cand;
    else if (q_ != hipErrorNotReady) return hip_fail(c, q_, "hipEventQuery(stage)");
  }
  if (k < 0) {
    k = sp.next;
    hipError_t e = hipEventSynchronize(sp.copied[k]);
    if (e != hipSuccess) return hip_fail(c, e, "hipEventSynchronize(stage)");
  }
  sp.next = (k + 1) % kStaticStages;
  unsigned char* h = static_cast<unsigned char*>(sp.stage[k]);
  std::memcpy(h, reqs, sizeof(bs_req_desc) * n);
  if (n_items) attention_items_into(reinterpret_cast<AttnItem*>(h + items_off), sp.tmp.get(), reqs, n, L, Hq, Hkv);
  const int meta[6] = {0, (int)items_off, (int)n_items, 0, 0, 0};   // whole rows: no merge list
  hipError_t e = hipMemcpyAsync(dscratch, h, blob_bytes, hipMemcpyHostToDevice, s);
  if (e != hipSuccess) return hip_fail(c, e, "hipMemcpyAsync(scratch)");
  e = hipEventRecord(sp.copied[k], s);
  if (e != hipSuccess) return hip_fail(c, e, "hipEventRecord(stage)");
  e = step_launch(c, dscratch, meta, n, L, R, W, n_layers, Hq, Hkv, D, dt, scale, write_back, q, k_new, v_new,
                  k_cache, v_cache, out, V, logits_dt, logits, logits_row_stride, tokens, tokens_row_stride, masked,
                  masked_row_stride, tau, q_min, eos_id, n_unmasked, done, eos_seen, conf_out, pos_out,
                  dscratch + kStaticBlobBytes, nullptr, s);
  if (e != hipSuccess) return hip_fail(c, e, "no-alloc step launch");
  return BS_OK;
}

int bs_profile_begin(bs_ctx* c, int max_steps) {
  if (!c) return fail(nullptr, BS_ERR_INVALID_ARG, "ctx is NULL");
  if (max_steps < 1 || max_steps > 1 << 16) return fail(c, BS_ERR_INVALID_ARG, "max_steps=%d outside [1, 65536]", max_steps);
  DeviceGuard dg(c->device);
  if (!dg.ok) return fail(c, BS_ERR_HIP, "hipSetDevice(%d) failed", c->device);
  Prof& p = c->prof;
  const size_t need = (size_t)max_steps * (kProfPhases + 1);
  while (p.ev.size() < need) {
    // timing-only events: no system-scope fence (cache write-back and
    // invalidate) at each mark, which would otherwise be charged to the phases
    hipEvent_t e = nullptr;
    hipError_t r = hipEventCreateWithFlags(&e, hipEventDisableSystemFence);
    if (r != hipSuccess) return hip_fail(c, r, "hipEventCreate(profile)");
    p.ev.push_back(e);
  }
  p.cap = max_steps;
  p.used = 0;
  p.on = true;
  return BS_OK;
}

int bs_profile_end(bs_ctx* c, float* phase_ms, int max_steps, int* n_steps) {
  if (!c) return fail(nullptr, BS_ERR_INVALID_ARG, "ctx is NULL");
  if (!n_steps || (max_steps > 0 && !phase_ms)) return fail(c, BS_ERR_INVALID_ARG, "output pointer is NULL");
  Prof& p = c->prof;
  if (!p.on) return fail(c, BS_ERR_INVALID_ARG, "profiling was not started");
  p.on = false;
  DeviceGuard dg(c->device);
  if (!dg.ok) return fail(c, BS_ERR_HIP, "hipSetDevice(%d) failed", c->device);
  const int m = std::min(p.used, std::max(max_steps, 0));
  for (int k = 0; k < m; ++k) {
    hipEvent_t* ev = &p.ev[(size_t)k * (kProfPhases + 1)];
    hipError_t r = hipEventSynchronize(ev[kProfPhases]);
    if (r != hipSuccess) return hip_fail(c, r, "hipEventSynchronize(profile)");
    for (int ph = 0; ph < kProfPhases; ++ph) {
      float ms = 0.0f;
      r = hipEventElapsedTime(&ms, ev[ph], ev[ph + 1]);
      if (r != hipSuccess) return hip_fail(c, r, "hipEventElapsedTime(profile)");
      phase_ms[(size_t)k * kProfPhases + ph] = ms;
    }
  }
  *n_steps = m;
  return BS_OK;
}

// ------------------------------------------------------------------ K4
int bs_kv_scatter_compact(bs_ctx* c, const bs_copy_seg* segs, int nseg, int n_layers, int Hkv,
                          int D, bs_dtype dt, const void* src_k, const void* src_v,
                          int64_t src_layer_stride, int R_src, int W_src, const void* stg_k,
                          const void* stg_v, int64_t stg_layer_stride, int R_stg, int W_stg,
                          void* dst_k, void* dst_v, int64_t dst_layer_stride, int R_dst, int W_dst,
                          void* stream) {
  if (!c) return fail(nullptr, BS_ERR_INVALID_ARG, "ctx is NULL");
  const int eb = dtype_bytes(dt);
  if (!eb) return fail(c, BS_ERR_INVALID_ARG, "bad dtype %d", (int)dt);
  if (nseg < 0 || n_layers < 0 || Hkv < 1 || D < 1) return fail(c, BS_ERR_INVALID_ARG, "negative or zero size");
  if (nseg > 0 && !segs) return fail(c, BS_ERR_INVALID_ARG, "segs is NULL");
  const int64_t row_bytes = (int64_t)D * eb;
  if (row_bytes % 16) return fail(c, BS_ERR_UNSUPPORTED, "D*elem=%lld not a multiple of 16 bytes", (long long)row_bytes);
  bool any_src = false, any_stg = false;
  for (int i = 0; i < nseg; ++i) (segs[i].src_kind ? any_stg : any_src) = true;
  const bool src_alias = any_src && (src_k == dst_k || src_v == dst_v || src_k == dst_v || src_v == dst_k);
  const bool stg_alias = any_stg && (stg_k == dst_k || stg_v == dst_v || stg_k == dst_v || stg_v == dst_k);
  int st = check_segments(c, segs, nseg, R_src, W_src, R_stg, W_stg, R_dst, W_dst, src_alias, stg_alias);
  if (st) return st;
  int64_t total_chunks = 0;
  for (int i = 0; i < nseg; ++i) total_chunks += (segs[i].len * row_bytes + kCopyChunkBytes - 1) / kCopyChunkBytes;
  if (any_src && (!src_k || !src_v)) return fail(c, BS_ERR_INVALID_ARG, "src box is NULL");
  if (any_stg && (!stg_k || !stg_v)) return fail(c, BS_ERR_INVALID_ARG, "staging box is NULL");
  if (nseg > 0 && (!dst_k || !dst_v)) return fail(c, BS_ERR_INVALID_ARG, "dst box is NULL");
  auto box_ok = [&](int64_t ls, int Rb, int Wb) { return ls >= (int64_t)Rb * Hkv * Wb * row_bytes && ls % 16 == 0; };
  if ((any_src && !box_ok(src_layer_stride, R_src, W_src)) || (any_stg && !box_ok(stg_layer_stride, R_stg, W_stg)) ||
      (nseg > 0 && !box_ok(dst_layer_stride, R_dst, W_dst)))
    return fail(c, BS_ERR_INVALID_ARG, "layer stride smaller than one box or not a multiple of 16 bytes");
  for (const void* p : {src_k, src_v, stg_k, stg_v, (const void*)dst_k, (const void*)dst_v})
    if (p && !aligned(p, 16)) return fail(c, BS_ERR_INVALID_ARG, "box pointers must be 16-byte aligned");
  if (nseg == 0 || n_layers == 0 || total_chunks == 0) return BS_OK;
  DeviceGuard dg(c->device);
  if (!dg.ok) return fail(c, BS_ERR_HIP, "hipSetDevice(%d) failed", c->device);
  hipStream_t s = static_cast<hipStream_t>(stream);
  Slot* sl = nullptr;
  st = upload(c, s, Key('C', {nseg, row_bytes}, segs, sizeof(bs_copy_seg) * nseg), [&](Blob& blob) {
    std::vector<CopyUnit> units;
    units.reserve((size_t)total_chunks);
    for (int i = 0; i < nseg; ++i) {
      const int64_t nc = (segs[i].len * row_bytes + kCopyChunkBytes - 1) / kCopyChunkBytes;
      for (int64_t k = 0; k < nc; ++k) units.push_back(CopyUnit{i, (int32_t)k});
    }
    blob.meta[0] = (int)blob.add(segs, sizeof(bs_copy_seg) * nseg);
    blob.meta[1] = (int)blob.add(units.data(), sizeof(CopyUnit) * units.size());
    blob.meta[2] = (int)units.size();
  }, &sl);
  if (st) return st;
  const char* base = static_cast<const char*>(sl->d);
  CopyArgs a{};
  a.segs = reinterpret_cast<const bs_copy_seg*>(base + sl->meta[0]);
  a.units = reinterpret_cast<const CopyUnit*>(base + sl->meta[1]);
  a.n_units = sl->meta[2];
  a.n_layers = n_layers; a.Hkv = Hkv; a.row_bytes = row_bytes;
  a.src_k = static_cast<const char*>(src_k); a.src_v = static_cast<const char*>(src_v);
  a.src_ls = src_layer_stride; a.W_src = W_src;
  a.stg_k = static_cast<const char*>(stg_k); a.stg_v = static_cast<const char*>(stg_v);
  a.stg_ls = stg_layer_stride; a.W_stg = W_stg;
  a.dst_k = static_cast<char*>(dst_k); a.dst_v = static_cast<char*>(dst_v);
  a.dst_ls = dst_layer_stride; a.W_dst = W_dst;
  hipError_t e = launch_compact(a, s);
  return finish(c, sl, s, e, "compact launch");
}

}  // extern "C"
