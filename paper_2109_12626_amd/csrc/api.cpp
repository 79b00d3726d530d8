// C ABI of libdpar: argument checks, plan cache, pointer-table staging and
// executor dispatch (Traeff 2021, Section 1 problem statement; Algorithm 1).
#include <hip/hip_runtime_api.h>

#include <algorithm>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <map>
#include <memory>
#include <mutex>
#include <string>
#include <vector>

#include "dpar.h"
#include "kernels.hpp"
#include "plan.hpp"

namespace {

thread_local std::string g_err;
thread_local hipEvent_t g_phase_event = nullptr;

int fail(int code, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
int fail(int code, const char* fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_err = buf;
  return code;
}

int hip_fail(hipError_t e, const char* what) {
  return fail(DPAR_ERR_HIP, "%s: %s", what, hipGetErrorString(e));
}

constexpr int kCounterSlots = 64;      // concurrent calls before reuse
using dpar::kCounterStride;            // uint32 words: 128-byte lines
// per call slot: kTicketCounters ticket lines, as many done-counter lines,
// then one line for the grid-barrier words
constexpr int kLinesPerSlot = 2 * dpar::kTicketCounters + 1;
constexpr int kStageSlots = 8;
// Retired pointer tables kept before one device-wide synchronisation frees
// them all (a restage does not wait for the calls that read the table).
constexpr size_t kRetiredTables = 32;
// Split executor, post-order work items: workgroups resident per CU in the
// up-phase (4 of 2 wavefronts read p = 1152 rows about 1.4% faster than the
// 8 that fit by LDS), applied from kCapMinRanks ranks and kCapMinItemsPerCu
// work items per CU on.
constexpr int kSeqWgPerCu = 4;
constexpr int kCapMinRanks = 256;
constexpr int kCapMinItemsPerCu = 64;
// Subtree work items: the deep load pipeline from this many ranks on.
constexpr int kSubDeepMinRanks = 1024;
// AUTO: a call of wide work items runs as one fused launch with at most
// kWideFuseAnyRanks ranks, with at most kWideFuseTwoRanks ranks and at most
// two items per CU (then without tail items), or with at most
// kWideFuseMaxRanks ranks and at most one item per CU.
constexpr int kWideFuseMaxRanks = 36;
constexpr int kWideFuseTwoRanks = 20;
constexpr int kWideFuseAnyRanks = 8;
// Wide work items from 3/4 of an item per CU on, from 7/8 with at most
// kWideLateRanks ranks.
constexpr int kWideLateRanks = 16;
// AUTO: level work items run split from kLvSplitRanks ranks on, and from
// kLvSplitManyRanks on with at least one item per CU, else fused; from
// kLvCrowdRanks ranks on they are taken up to four per CU before subtree
// items (else two).
constexpr int kLvSplitRanks = 1024;
constexpr int kLvSplitManyRanks = 512;
constexpr int kLvCrowdRanks = 2048;
// Ranks from which subtree items take calls of up to four items per CU.
constexpr int kSubCrowdRanks = 4096;
// Level work item: loads in flight at once (1024 threads, 8 loads each).
constexpr uint64_t kLvLoadsInFlight = 1024 * 8;
// Ticket executor: rank loads per claimed batch of work items.
constexpr uint64_t kTicketRankLoads = 1024;
// Largest p whose post-order work items use one wavefront for both trees.
constexpr int kOneWaveMaxRanks = 48;
// Calls that leave trailing elements after the last 4-element quantum and
// move at most this many bytes (2 p m times the element size) take one
// element per lane in one launch instead of 16-byte lanes plus a launch for
// the trailing elements (measured, int32 SUM, b = 1: p = 288, m = 8750
// (20 MB) 20.4 vs 28.1 us; m = 21250 (49 MB) 35.8 vs 32.6 us; p = 1152,
// m = 2125 (20 MB) 34.7 vs 38.1 us; m = 8750 (81 MB) 66.0 vs 59.0 us).
constexpr uint64_t kScalarBelowBytes = 24ull << 20;
// Split executor's broadcast pass: y_0 is streamed out in spans of at most
// this many KB (2 MB per XCD's 4 MB L2; a 32 MB y_0 taken as one span ran at
// half the speed).
constexpr int kBcastSpanKB = 16384;
// The broadcast pass finds each workgroup's row and tile by multiplication
// (plan.hpp fastdiv) when it writes at most this many bytes, else by
// division (two instantiations of the pass).  Measured against division,
// split executor, cold caches: p = 1152, m = 2^16 int32 (0.3 GB written)
// 72 -> 69 us; p = 36, m = 2^20 31.3 -> 29.8 us; the 64-rank matrix product
// 48.3 -> 46.4 us; at p = 1152, m = 2^22 fp32 (19 GB, warm) division is the
// faster one (2.65 against 2.73 ms).
constexpr uint64_t kBcastFastDivMaxBytes = 2ull << 30;

struct OpsTable {
  uint32_t* dev = nullptr;   // opcodes, padded
  uint32_t* lvl = nullptr;   // level-ordered entries + boundaries (p <= 65534)
  uint32_t* dn = nullptr;    // parent << 8 | depth of the real tree(s)
  uint32_t* dord = nullptr;  // depth offsets + non-root ranks by depth
  uint32_t* sub = nullptr;   // subtree work-item plan (null: not available)
  int sub_ns = 0;            // its slots per wavefront
  std::vector<uint32_t> doff;  // the depth offsets, host copy
  int height = 0;              // of the kernel form
  int real_height = 0;         // of the real tree(s)
  int n_a = 0;
  int root_a = -1, root_b = -1;  // roots of the real tree(s)
};

// A staged pointer set.  Its device table is never overwritten while it is
// staged: restaging the slot retires the table (kernels of earlier calls,
// on any stream, may still read it) and takes another from the pool, so no
// call needs to record anything to protect it.  The one event, recorded
// after each staging copy, guards the pinned source of that copy and orders
// the copy before calls on other streams.
struct StageSlot {
  std::vector<uint64_t> key;  // x pointers then y pointers
  uint64_t* host = nullptr;   // pinned: the staging copy's source
  size_t host_cap = 0;        // its entries
  uint64_t* dev = nullptr;    // the device table the kernels read
  size_t cap = 0;             // its entries
  hipEvent_t ev = nullptr;    // recorded after the staging copy
  hipStream_t copy_stream = nullptr;  // the stream that copy went on
  bool copy_pending = false;  // that copy may not have run yet
  bool pinned = false;        // read by a captured graph: never restaged
  unsigned long long last_use = 0;
};

// Device pointer tables not held by a slot: free ones may be written, retired
// ones may still be read by kernels already enqueued; all of those finish
// before the next device-wide synchronisation, after which a retired table
// is free.
struct TableBuf {
  uint64_t* dev;
  size_t cap;  // entries
};

struct DeviceState {
  int device = -1;
  int num_cus = 0;
  int lds_limit = 65536;         // dynamic LDS bytes per workgroup
  int lds_per_cu = 65536;        // LDS bytes per CU
  unsigned* counters = nullptr;  // kCounterSlots slots + one error line
  unsigned next_counter = 0;
  std::map<std::pair<int, int>, OpsTable> ops;  // (p, one tree?)
  StageSlot stage[kStageSlots];
  unsigned long long tick = 0;
  std::vector<TableBuf> free_tables;
  std::vector<TableBuf> retired_tables;
};

std::mutex g_mu;
std::map<int, std::unique_ptr<DeviceState>> g_devices;

// The allocation-free entry point (dpar_allreduce_noalloc): per device, the
// address of the library's fixed scratch array and what it holds.  Layout
// for p ranks: opcode table | level table | subtree plan | pointer tables,
// each at a 256-byte boundary.
constexpr int kFixedMaxDevices = 64;
struct FixedState {
  bool ready = false;
  DeviceState info;               // device attributes only: no counters,
                                  // tables or staging slots
  unsigned char* scratch = nullptr;  // this device's fixed scratch array
  int tables_p = 0;               // p whose tables the scratch holds (0: none)
  OpsTable ops;                   // device pointers into the scratch
  size_t ptr_off = 0;             // offset of the pointer tables
  std::vector<uint64_t> ptr_key;  // x then y pointers the scratch holds
};
FixedState g_fixed[kFixedMaxDevices];

int env_int(const char* name, int dflt) {
  const char* v = std::getenv(name);
  return v && *v ? std::atoi(v) : dflt;
}

unsigned long long spin_limit() {
  const char* v = std::getenv("DPAR_SPIN_LIMIT");
  return v && *v ? std::strtoull(v, nullptr, 10) : (1ull << 26);
}

int get_state(DeviceState** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  auto it = g_devices.find(dev);
  if (it != g_devices.end()) {
    *out = it->second.get();
    return DPAR_SUCCESS;
  }
  auto st = std::make_unique<DeviceState>();
  st->device = dev;
  e = hipDeviceGetAttribute(&st->num_cus, hipDeviceAttributeMultiprocessorCount,
                            dev);
  if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
  e = hipDeviceGetAttribute(&st->lds_limit,
                            hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
  if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
  e = hipDeviceGetAttribute(
      &st->lds_per_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor, dev);
  if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
  const size_t words =
      ((size_t)kCounterSlots * kLinesPerSlot + 1) * kCounterStride;
  e = hipMalloc(&st->counters, words * sizeof(unsigned));
  if (e != hipSuccess) return fail(DPAR_ERR_NOMEM, "counters: %s",
                                   hipGetErrorString(e));
  e = hipMemset(st->counters, 0, words * sizeof(unsigned));
  if (e != hipSuccess) return hip_fail(e, "hipMemset");
  *out = st.get();
  g_devices[dev] = std::move(st);
  return DPAR_SUCCESS;
}

template <class T>
int upload(const std::vector<T>& v, T** out, const char* what) {
  hipError_t e = hipMalloc(out, v.size() * sizeof(T));
  if (e != hipSuccess)
    return fail(DPAR_ERR_NOMEM, "%s: %s", what, hipGetErrorString(e));
  e = hipMemcpy(*out, v.data(), v.size() * sizeof(T), hipMemcpyHostToDevice);
  if (e != hipSuccess) {
    (void)hipFree(*out);
    *out = nullptr;
    return hip_fail(e, what);
  }
  return DPAR_SUCCESS;
}

void free_ops(OpsTable& t) {
  if (t.dev) (void)hipFree(t.dev);
  if (t.lvl) (void)hipFree(t.lvl);
  if (t.dn) (void)hipFree(t.dn);
  if (t.dord) (void)hipFree(t.dord);
  if (t.sub) (void)hipFree(t.sub);
  t.dev = t.lvl = t.dn = t.dord = t.sub = nullptr;
}

// Device tables for p ranks on the dual-root trees or on one tree: the
// opcodes and level table of the form the kernels evaluate, and the real
// tree's parents and depths for the round-structured down-step.
int get_ops(DeviceState* st, int p, bool single, const OpsTable** out) {
  const auto key = std::make_pair(p, single ? 1 : 0);
  auto it = st->ops.find(key);
  if (it != st->ops.end()) {
    *out = &it->second;
    return DPAR_SUCCESS;
  }
  const dpar::Tree kt = single ? dpar::kernel_single_tree(p)
                               : dpar::build_tree(p);
  const dpar::Tree real = single ? dpar::build_single_tree(p) : kt;
  OpsTable tab;
  tab.height = kt.height;
  tab.n_a = kt.n_a;
  tab.root_a = real.root_a;
  tab.root_b = real.root_b;
  tab.real_height = real.height;
  std::vector<uint32_t> ops = dpar::make_ops(kt);
  std::vector<uint32_t> sub;
  // the subtree work item cuts each tree two levels below its root
  const bool has_sub = p >= 64 && dpar::make_sub(kt, ops, 2, &sub);
  ops.resize(ops.size() + dpar::kTablePad, 0u);  // kernels read ahead
  int rc = upload(ops, &tab.dev, "opcode table");
  if (!rc && has_sub) {
    rc = upload(sub, &tab.sub, "subtree plan");
    tab.sub_ns = (int)sub[3];
  }
  if (!rc && p <= 65534) rc = upload(dpar::make_levels(kt), &tab.lvl,
                                     "level table");
  if (!rc && p < (1 << 24) && real.height < 256) {
    rc = upload(dpar::make_down(real), &tab.dn, "parent table");
    const std::vector<uint32_t> dord = dpar::make_depth_order(real);
    if (!rc) rc = upload(dord, &tab.dord, "depth order table");
    tab.doff.assign(dord.begin(), dord.begin() + real.height + 2);
  }
  if (rc) {
    free_ops(tab);
    return rc;
  }
  st->ops[key] = tab;
  *out = &st->ops[key];
  return DPAR_SUCCESS;
}

// Pointer sets (x then y) that passed the aliasing rules, with their row
// length in bytes; a few recent ones, most recent first.
struct AliasOk {
  std::vector<uint64_t> key;
  size_t bytes;
};
std::vector<AliasOk> g_alias_ok;

// The key holds the two arrays' pointer values as they are (8 bytes each),
// so whole arrays compare with memcmp (p = 1152: two 9 KB compares).
static_assert(sizeof(void*) == sizeof(uint64_t), "64-bit pointers");
bool same_key(const std::vector<uint64_t>& k, const void* const* x,
              void* const* y, int p) {
  if (k.size() != 2 * (size_t)p) return false;
  return std::memcmp(k.data(), x, (size_t)p * sizeof(uint64_t)) == 0 &&
         std::memcmp(k.data() + p, y, (size_t)p * sizeof(uint64_t)) == 0;
}

bool alias_cached(const void* const* x, void* const* y, int p, size_t bytes) {
  for (const AliasOk& a : g_alias_ok)
    if (a.bytes == bytes && same_key(a.key, x, y, p)) return true;
  return false;
}

void alias_remember(const void* const* x, void* const* y, int p,
                    size_t bytes) {
  AliasOk a;
  a.bytes = bytes;
  a.key.resize(2 * (size_t)p);
  for (int i = 0; i < p; ++i) {
    a.key[i] = (uint64_t)(uintptr_t)x[i];
    a.key[p + i] = (uint64_t)(uintptr_t)y[i];
  }
  g_alias_ok.insert(g_alias_ok.begin(), std::move(a));
  if (g_alias_ok.size() > 8) g_alias_ok.pop_back();
}

// A staging slot that already holds exactly these pointer arrays, if any.
bool find_staged(DeviceState* st, const void* const* x, void* const* y, int p,
                 StageSlot** out) {
  for (auto& s : st->stage) {
    if (s.dev && same_key(s.key, x, y, p)) {
      s.last_use = ++st->tick;
      *out = &s;
      return true;
    }
  }
  return false;
}

// A device table of at least `need` entries: a free one, else (with
// kRetiredTables retired) the retired ones once every kernel has finished,
// else a new allocation.
int take_table(DeviceState* st, size_t need, TableBuf* out) {
  auto fit = [&](std::vector<TableBuf>& v) {
    for (size_t i = 0; i < v.size(); ++i) {
      if (v[i].cap >= need) {
        *out = v[i];
        v.erase(v.begin() + (long)i);
        return true;
      }
    }
    return false;
  };
  if (fit(st->free_tables)) return DPAR_SUCCESS;
  hipError_t e;
  if (st->retired_tables.size() >= kRetiredTables) {
    e = hipDeviceSynchronize();
    if (e != hipSuccess) return hip_fail(e, "hipDeviceSynchronize");
    for (const TableBuf& t : st->retired_tables) {
      if (st->free_tables.size() < kRetiredTables)
        st->free_tables.push_back(t);
      else
        (void)hipFree(t.dev);
    }
    st->retired_tables.clear();
    if (fit(st->free_tables)) return DPAR_SUCCESS;
  }
  // the kernels read a few entries past the last pointer
  const size_t cap = std::max<size_t>(need, 512 + dpar::kTablePad);
  out->cap = cap;
  e = hipMalloc(&out->dev, cap * sizeof(uint64_t));
  if (e != hipSuccess) return fail(DPAR_ERR_NOMEM, "pointer table: %s",
                                   hipGetErrorString(e));
  return DPAR_SUCCESS;
}

// Copies the two pointer arrays into the least recently used staging slot
// (callers look for a slot holding the same arrays first).
int stage_pointers(DeviceState* st, const void* const* x, void* const* y,
                   int p, hipStream_t stream, StageSlot** used) {
  std::vector<uint64_t> key(2 * (size_t)p);
  for (int i = 0; i < p; ++i) {
    key[i] = (uint64_t)(uintptr_t)x[i];
    key[p + i] = (uint64_t)(uintptr_t)y[i];
  }
  ++st->tick;
  StageSlot* s = nullptr;
  for (auto& c : st->stage)
    if (!c.pinned && (!s || c.last_use < s->last_use)) s = &c;
  if (!s)
    return fail(DPAR_ERR_NOMEM, "every pointer staging slot is held by a "
                                "captured graph (dpar_finalize releases them)");
  hipError_t e;
  if (s->copy_pending) {  // its pinned source is rewritten below
    e = hipEventSynchronize(s->ev);
    if (e != hipSuccess) return hip_fail(e, "hipEventSynchronize");
    s->copy_pending = false;
  }
  if (s->dev) {  // earlier calls may still read it
    st->retired_tables.push_back(TableBuf{s->dev, s->cap});
    s->dev = nullptr;
    s->cap = 0;
  }
  s->key.clear();
  const size_t need = key.size() + dpar::kTablePad;
  if (s->host_cap < key.size()) {
    if (s->host) (void)hipHostFree(s->host);
    s->host = nullptr;
    s->host_cap = 0;
    const size_t hcap = std::max<size_t>(key.size(), 512);
    e = hipHostMalloc(&s->host, hcap * sizeof(uint64_t), hipHostMallocDefault);
    if (e != hipSuccess) return fail(DPAR_ERR_NOMEM, "pinned staging: %s",
                                     hipGetErrorString(e));
    s->host_cap = hcap;
  }
  TableBuf t{};
  int rc = take_table(st, need, &t);
  if (rc) return rc;
  s->dev = t.dev;
  s->cap = t.cap;
  if (!s->ev) {
    e = hipEventCreateWithFlags(&s->ev, hipEventDisableTiming);
    if (e != hipSuccess) return hip_fail(e, "hipEventCreate");
  }
  std::memcpy(s->host, key.data(), key.size() * sizeof(uint64_t));
  e = hipMemcpyAsync(s->dev, s->host, key.size() * sizeof(uint64_t),
                     hipMemcpyHostToDevice, stream);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpyAsync pointer table");
  e = hipEventRecord(s->ev, stream);
  if (e != hipSuccess) return hip_fail(e, "hipEventRecord");
  s->copy_pending = true;
  s->copy_stream = stream;
  s->key = std::move(key);
  s->last_use = st->tick;
  *used = s;
  return DPAR_SUCCESS;
}

// A call on `stream` about to read slot s's table: the staging copy, if it
// may not have run yet and went on another stream, goes before this call's
// kernels (a wait on the device; on the host under capture, whose stream
// cannot wait for work outside the graph).
int order_after_copy(StageSlot* s, hipStream_t stream, bool capturing) {
  if (!s->copy_pending || s->copy_stream == stream) return DPAR_SUCCESS;
  hipError_t e = hipEventQuery(s->ev);
  if (e == hipSuccess) {
    s->copy_pending = false;
    return DPAR_SUCCESS;
  }
  if (e != hipErrorNotReady) return hip_fail(e, "hipEventQuery");
  e = capturing ? hipEventSynchronize(s->ev)
                : hipStreamWaitEvent(stream, s->ev, 0);
  if (e != hipSuccess) return hip_fail(e, "waiting for the pointer staging");
  if (capturing) s->copy_pending = false;
  return DPAR_SUCCESS;
}

// The fixed scratch of the current device; its address is looked up once per
// device (with that device current) and kept.  Allocates nothing.
int get_fixed(FixedState** out) {
  int dev = 0;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  if (dev < 0 || dev >= kFixedMaxDevices)
    return fail(DPAR_ERR_UNSUPPORTED, "device %d beyond the fixed scratch "
                                      "table", dev);
  FixedState& f = g_fixed[dev];
  if (!f.ready) {
    DeviceState& st = f.info;
    st.device = dev;
    e = hipDeviceGetAttribute(&st.num_cus,
                              hipDeviceAttributeMultiprocessorCount, dev);
    if (e == hipSuccess)
      e = hipDeviceGetAttribute(&st.lds_limit,
                                hipDeviceAttributeMaxSharedMemoryPerBlock, dev);
    if (e == hipSuccess)
      e = hipDeviceGetAttribute(
          &st.lds_per_cu, hipDeviceAttributeMaxSharedMemoryPerMultiprocessor,
          dev);
    if (e != hipSuccess) return hip_fail(e, "hipDeviceGetAttribute");
    void* ptr = nullptr;
    e = dpar::fixed_scratch_address(&ptr);
    if (e != hipSuccess || !ptr)
      return hip_fail(e != hipSuccess ? e : hipErrorInvalidSymbol,
                      "hipGetSymbolAddress(fixed scratch)");
    f.scratch = static_cast<unsigned char*>(ptr);
    f.ready = true;
  }
  *out = &f;
  return DPAR_SUCCESS;
}

size_t align256(size_t v) { return (v + 255) & ~(size_t)255; }

// Device tables for p ranks (dual-root trees) in the fixed scratch, staged
// through kernel arguments on `stream` unless the scratch holds them already.
int fixed_tables(FixedState* f, int p, hipStream_t stream,
                 const OpsTable** out) {
  if (f->tables_p == p) {
    *out = &f->ops;
    return DPAR_SUCCESS;
  }
  f->tables_p = 0;  // whatever follows, the old tables are gone
  f->ptr_key.clear();
  const dpar::Tree kt = dpar::build_tree(p);
  std::vector<uint32_t> ops = dpar::make_ops(kt);
  std::vector<uint32_t> sub;
  const bool has_sub = p >= 64 && dpar::make_sub(kt, ops, 2, &sub);
  ops.resize(ops.size() + dpar::kTablePad, 0u);  // kernels read ahead
  const std::vector<uint32_t> lvl = dpar::make_levels(kt);
  const size_t off_lvl = align256(ops.size() * 4);
  const size_t off_sub = off_lvl + align256(lvl.size() * 4);
  const size_t off_ptr = off_sub + align256(sub.size() * 4);
  const size_t ptr_bytes = (2 * (size_t)p + dpar::kTablePad) * 8;
  if (off_ptr + align256(ptr_bytes) > dpar::kFixedScratchBytes)
    return fail(DPAR_ERR_UNSUPPORTED, "p = %d: tables exceed the fixed "
                "scratch of %zu bytes", p, dpar::kFixedScratchBytes);
  unsigned char* base = f->scratch;
  hipError_t e = dpar::stage_by_args(base, ops.data(), ops.size() * 4, stream);
  if (e == hipSuccess)
    e = dpar::stage_by_args(base + off_lvl, lvl.data(), lvl.size() * 4,
                            stream);
  if (e == hipSuccess && has_sub)
    e = dpar::stage_by_args(base + off_sub, sub.data(), sub.size() * 4,
                            stream);
  if (e != hipSuccess) return hip_fail(e, "staging the tables");
  OpsTable t;
  t.dev = reinterpret_cast<uint32_t*>(base);
  t.lvl = reinterpret_cast<uint32_t*>(base + off_lvl);
  t.sub = has_sub ? reinterpret_cast<uint32_t*>(base + off_sub) : nullptr;
  t.sub_ns = has_sub ? (int)sub[3] : 0;
  t.height = kt.height;
  t.real_height = kt.height;
  t.n_a = kt.n_a;
  t.root_a = kt.root_a;
  t.root_b = kt.root_b;
  f->ops = t;
  f->ptr_off = off_ptr;
  f->tables_p = p;
  *out = &f->ops;
  return DPAR_SUCCESS;
}

// The pointer tables in the fixed scratch (after fixed_tables for this p).
int fixed_pointers(FixedState* f, const void* const* x, void* const* y,
                   int p, hipStream_t stream, const uint64_t** out) {
  uint64_t* dev = reinterpret_cast<uint64_t*>(f->scratch + f->ptr_off);
  if (!same_key(f->ptr_key, x, y, p)) {
    f->ptr_key.clear();
    std::vector<uint64_t> key(2 * (size_t)p + dpar::kTablePad, 0u);
    for (int i = 0; i < p; ++i) {
      key[i] = (uint64_t)(uintptr_t)x[i];
      key[p + i] = (uint64_t)(uintptr_t)y[i];
    }
    const hipError_t e =
        dpar::stage_by_args(dev, key.data(), key.size() * 8, stream);
    if (e != hipSuccess) return hip_fail(e, "staging the pointer tables");
    key.resize(2 * (size_t)p);
    f->ptr_key = std::move(key);
  }
  *out = dev;
  return DPAR_SUCCESS;
}

size_t elem_size(dpar_dtype_t dt) { return dt == DPAR_U32_MAT2X2 ? 16 : 4; }

bool valid_pair(dpar_dtype_t dt, dpar_op_t op) {
  return (dt == DPAR_INT32 && (op == DPAR_SUM || op == DPAR_MAX)) ||
         (dt == DPAR_FLOAT32 && op == DPAR_SUM) ||
         (dt == DPAR_U32_MAT2X2 && op == DPAR_MATMUL);
}

dpar::Kind kind_of(dpar_dtype_t dt, dpar_op_t op) {
  if (dt == DPAR_U32_MAT2X2) return dpar::Kind::MAT;
  if (dt == DPAR_FLOAT32) return dpar::Kind::F32_SUM;
  return op == DPAR_MAX ? dpar::Kind::I32_MAX : dpar::Kind::I32_SUM;
}

// Output ranges must be pairwise disjoint; an output range may coincide
// exactly with an input range (in place) but not overlap one partially.  All
// 2p ranges have the same length, so two of them overlap exactly when their
// start addresses differ by less than that length.
bool aliasing_ok(const void* const* x, void* const* y, int p, size_t bytes) {
  if (bytes == 0) return true;
  std::vector<uint64_t> in(p), out(p);
  for (int i = 0; i < p; ++i) {
    in[i] = (uint64_t)(uintptr_t)x[i];
    out[i] = (uint64_t)(uintptr_t)y[i];
  }
  std::sort(in.begin(), in.end());
  std::sort(out.begin(), out.end());
  for (int i = 1; i < p; ++i)
    if (out[i] - out[i - 1] < bytes) return false;
  for (uint64_t lo : out) {
    const uint64_t from = lo >= bytes ? lo - bytes + 1 : 0;
    auto first = std::lower_bound(in.begin(), in.end(), from);
    auto last = std::lower_bound(in.begin(), in.end(), lo + bytes);
    for (auto it = first; it != last; ++it)
      if (*it != lo) return false;
  }
  return true;
}

}  // namespace

extern "C" {

const char* dpar_last_error(void) { return g_err.c_str(); }

int dpar_set_phase_event(hipEvent_t ev) {
  g_err.clear();
  g_phase_event = ev;
  return DPAR_SUCCESS;
}

int dpar_tree_info(int p, int rank, dpar_node_t* out) {
  g_err.clear();
  if (p < 1 || rank < 0 || rank >= p || !out)
    return fail(DPAR_ERR_INVALID_ARG, "dpar_tree_info: bad p/rank/out");
  const dpar::Tree t = dpar::build_tree(p);
  out->parent = t.parent[rank];
  out->child0 = t.child0[rank];
  out->child1 = t.child1[rank];
  out->depth = t.depth[rank];
  out->subtree_lo = t.lo[rank];
  out->dual = t.dual[rank];
  return DPAR_SUCCESS;
}

int dpar_tree_info_alg(int p, dpar_alg_t alg, int rank, dpar_node_t* out) {
  g_err.clear();
  if (alg < DPAR_ALG_DUAL_ROOT || alg > DPAR_ALG_REDUCE_BCAST)
    return fail(DPAR_ERR_INVALID_ARG, "dpar_tree_info_alg: unknown alg %d",
                (int)alg);
  if (alg == DPAR_ALG_DUAL_ROOT) return dpar_tree_info(p, rank, out);
  if (p < 1 || rank < 0 || rank >= p || !out)
    return fail(DPAR_ERR_INVALID_ARG, "dpar_tree_info_alg: bad p/rank/out");
  const dpar::Tree t = dpar::build_single_tree(p);
  out->parent = t.parent[rank];
  out->child0 = t.child0[rank];
  out->child1 = t.child1[rank];
  out->depth = t.depth[rank];
  out->subtree_lo = t.lo[rank];
  out->dual = -1;
  return DPAR_SUCCESS;
}

int dpar_schedule_rounds(int p, int b, dpar_alg_t alg) {
  g_err.clear();
  if (p < 1 || b < 1)
    return fail(DPAR_ERR_INVALID_ARG, "dpar_schedule_rounds: bad p/b");
  if (alg < DPAR_ALG_DUAL_ROOT || alg > DPAR_ALG_REDUCE_BCAST)
    return fail(DPAR_ERR_INVALID_ARG, "dpar_schedule_rounds: unknown alg");
  const dpar::Tree t = alg == DPAR_ALG_DUAL_ROOT ? dpar::build_tree(p)
                                                 : dpar::build_single_tree(p);
  const long long r =
      alg == DPAR_ALG_REDUCE_BCAST
          ? (t.height > 0 ? 2ll * b + t.height - 1 : (long long)b)
          : (long long)b + t.height;
  if (r > 2147483647ll)
    return fail(DPAR_ERR_UNSUPPORTED, "dpar_schedule_rounds: too many rounds");
  return (int)r;
}

int dpar_block_rule(int p, size_t m, double alpha, double beta) {
  g_err.clear();
  if (p < 1) return fail(DPAR_ERR_INVALID_ARG, "dpar_block_rule: p < 1");
  return (int)dpar::block_rule(p, m, alpha, beta);
}

int dpar_rounds(int p, int b, int rank) {
  g_err.clear();
  if (p < 1 || b < 1 || rank < -1 || rank >= p)
    return fail(DPAR_ERR_INVALID_ARG, "dpar_rounds: bad p/b/rank");
  return dpar::rank_rounds(dpar::build_tree(p), b, rank);
}

// Wavefronts per post-order work item: one per tree, except for small trees
// (p <= kOneWaveMaxRanks), where one wavefront walking both trees is faster
// (measured for int32 SUM and the matrix product at 256 MB and 1 GB per
// side: p = 4..48 up to 27% faster, equal from 64 to 192, slower at 512).
// DPAR_WAVES=1|2 overrides.
int chunk_waves(int p) {
  if (p < 2) return 1;
  const int w = env_int("DPAR_WAVES", p <= kOneWaveMaxRanks ? 1 : 2);
  return w == 1 ? 1 : 2;
}

// One element per lane (see allreduce_impl).
static bool one_element_per_lane(int p, size_t m, dpar_dtype_t dtype,
                                 bool rounds_exec) {
  if (env_int("DPAR_SCALAR", 0) != 0) return true;
  if (m % 4 == 0 || dtype == DPAR_U32_MAT2X2) return false;
  return rounds_exec ||
         2ull * (uint64_t)p * m * elem_size(dtype) <= kScalarBelowBytes;
}

// Vector path (16-byte lanes: 4 scalars or one matrix) whenever the blocks
// hold whole quanta; rows need only the 4-byte alignment every call requires
// (16-byte accesses at 4-byte aligned addresses: at p = 1152, m = 2^22 int32
// with rows 4 bytes off a 16-byte boundary 7.0 ms per call, against 16.4 ms
// with one element per lane).  Blocks are cut at lines of 8 quanta (128
// bytes on 16-byte aligned rows) when there are at least b lines, else at
// quanta.  Otherwise (int32/fp32 blocks shorter than 4 elements, or
// one_per_lane) one element per lane and the canonical element partition.
static void choose_schedule(size_t m, dpar_dtype_t dtype, int b,
                            bool one_per_lane, dpar::Schedule* s,
                            dpar::Path* path) {
  *path = dpar::Path::SCALAR;
  int g = 1, lq = 1;
  if (dtype == DPAR_U32_MAT2X2) {
    *path = dpar::Path::VEC16;
    lq = (m + 7) / 8 >= (size_t)b ? 8 : 1;
  } else if (!one_per_lane && m / 4 >= (size_t)b) {
    *path = dpar::Path::VEC16;
    g = 4;
    lq = (m / 4 + 7) / 8 >= (size_t)b ? 8 : 1;
  }
  *s = dpar::make_schedule(m, b, g, lq);
}

int dpar_schedule_info(int p, size_t m, dpar_dtype_t dtype, int b, int aligned,
                       dpar_schedule_t* out) {
  g_err.clear();
  if (p < 1 || b < 0 || !out || m == 0)
    return fail(DPAR_ERR_INVALID_ARG, "dpar_schedule_info: bad arguments");
  if (dtype < DPAR_INT32 || dtype > DPAR_U32_MAT2X2)
    return fail(DPAR_ERR_UNSUPPORTED, "dpar_schedule_info: dtype");
  if (b == 0) b = (int)dpar::block_rule(p, m, 0.0, 0.0);
  if ((size_t)b > m) return fail(DPAR_ERR_INVALID_ARG, "b > m");
  dpar::Schedule s;
  dpar::Path path;
  (void)aligned;  // the decomposition does not depend on alignment
  choose_schedule(m, dtype, b, one_element_per_lane(p, m, dtype, false), &s,
                  &path);
  const dpar::Tree t = dpar::build_tree(p);
  out->b = s.b;
  out->granularity = s.g * s.lq;
  out->quantum = s.g;
  out->nquanta = s.Q;
  out->tail_elems = s.tail;
  out->chunks_per_block = s.C;
  out->height = t.height;
  out->waves_per_chunk = chunk_waves(p);
  return DPAR_SUCCESS;
}

int dpar_block_bounds(const dpar_schedule_t* s, size_t m, int j,
                      size_t* start, size_t* end) {
  g_err.clear();
  if (!s || !start || !end || j < 0 || j >= s->b || s->b < 1)
    return fail(DPAR_ERR_INVALID_ARG, "dpar_block_bounds: bad arguments");
  if (s->quantum < 1 || s->granularity % s->quantum)
    return fail(DPAR_ERR_INVALID_ARG, "dpar_block_bounds: bad schedule");
  dpar::Schedule sc = dpar::make_schedule(
      (uint64_t)s->nquanta * s->quantum, s->b, s->quantum,
      s->granularity / s->quantum);
  uint64_t qs, qe;
  dpar::block_quanta(sc, j, &qs, &qe);
  *start = (size_t)(qs * (uint64_t)s->quantum);
  *end = (size_t)(qe * (uint64_t)s->quantum);
  if (j == s->b - 1) *end = m;  // the tail rides with the last block
  return DPAR_SUCCESS;
}

}  // extern "C"

namespace {

// The device executor for a public one.  AUTO is the split executor, or,
// for calls moving at most DPAR_FUSE_BELOW_KB (default 40 MB), one launch of
// every work item in round order with the fused write-out (measured: 1-4 us
// faster up to 40 MB moved; from ~80 MB up it can be slower, e.g. p = 300,
// m = 2^15, b = 520: 51.7 vs 46.9 us).
dpar::Exec device_exec(dpar_exec_t exec, int p, uint64_t bytes_moved) {
  switch (exec) {
    case DPAR_EXEC_LAUNCH_PER_ROUND: return dpar::Exec::LAUNCH_PER_ROUND;
    case DPAR_EXEC_GRID_BARRIER: return dpar::Exec::GRID_BARRIER;
    case DPAR_EXEC_TICKET: return dpar::Exec::TICKET;
    case DPAR_EXEC_ROUNDS: return dpar::Exec::ROUNDS;
    case DPAR_EXEC_ROUNDS_BARRIER: return dpar::Exec::ROUNDS_BARRIER;
    case DPAR_EXEC_SPLIT:
      return p < 2 ? dpar::Exec::DISPATCH : dpar::Exec::SPLIT;
    default: break;
  }
  if (p < 2 || bytes_moved <= (uint64_t)env_int("DPAR_FUSE_BELOW_KB",
                                                40 * 1024) * 1024ull)
    return dpar::Exec::DISPATCH;
  return dpar::Exec::SPLIT;
}

// Work items of a one-launch run with groups of grp consecutive blocks.
uint64_t grouped_units(const dpar::Schedule& s, int grp) {
  return (((uint64_t)s.b + (uint64_t)grp - 1) / (uint64_t)grp) *
         (uint64_t)s.C;
}

// Blocks per work-item group.  The one-launch executors (split, ticket, one
// fused launch) issue the rounds' work items in round order from one
// launch, so a work item may carry several consecutive whole blocks: blocks
// shorter than half a chunk are grouped (plan.hpp block_group), else a
// wavefront of 64 lanes would carry as few as a handful of quanta.
// Per-round executors: 1.
int block_group(dpar::Exec ex, const dpar::Schedule& s) {
  const bool one_launch = ex == dpar::Exec::SPLIT ||
                          ex == dpar::Exec::DISPATCH ||
                          ex == dpar::Exec::TICKET;
  if (!one_launch || env_int("DPAR_GROUP_BLOCKS", 1) == 0) return 1;
  return dpar::block_group(s);
}

// The split up-phase's residency cap for post-order work items (at most
// kSeqWgPerCu workgroups per CU, set through the LDS request): long walks
// (p >= kCapMinRanks) and at least kCapMinItemsPerCu items per CU.
bool seq_wg_capped(int p, uint64_t items, const DeviceState& st) {
  return p >= kCapMinRanks &&
         items >= (uint64_t)kCapMinItemsPerCu * (uint64_t)st.num_cus;
}

// Longest rows (bytes) on which AUTO runs post-order items as one fused
// launch: 3.5 MB up to 16 ranks (where wide items take longer rows), 2.5 MB
// up to 48, 1.5 MB up to 64, 1 MB up to 96, 512 KB beyond (rows of 16 KB
// chunks: 224, 160, 96, 64, 32).
uint64_t seq_fuse_row_bytes(int p) {
  return p <= kWideLateRanks ? (7ull << 19)
         : p <= 48           ? (5ull << 19)
         : p <= 64           ? (3ull << 19)
         : p <= 96           ? (1ull << 20)
                             : (1ull << 19);
}

// Full wide items of a call of n wide chunks.  A wide item holds its CU for
// a chain of p / kWideKF dependent visits, so a last round of one item per
// CU with only a few items left leaves most CUs idle for about as long as
// a full round (int32 SUM, split, p = 288, up-phase: 256 items 178 us,
// 264 items 308 us, 519 items 483 us), and where two fit per CU by LDS
// (p <= 48) the CUs that get two finish late (p = 36: 256 items 60.3 us
// per call, 264 items 67.6 us).  The columns past the last whole round of
// one item per CU go instead to tail items with one quantum per lane and
// 8 visits in flight (p = 288: 211 and 387 us; p = 128, 264 items:
// 140 -> 97 us; p = 36, 264 items: 62.0 us per call), unless they fill
// more than 7/8 of a round, where the full items are as fast or faster
// (p = 288, 504 items: 353 us full, 363 us with tail items; p = 36:
// 102.0 vs 102.4 us per call; with 448 items tail items are faster: p = 128
// 152 -> 142 us, p = 36 94.5 -> 92.4 us per call).  DPAR_WIDE_TAIL=0: no
// tail items; DPAR_WIDE_ROUND: items per round (default: the CU count;
// tests: tail items on small calls).
uint64_t wide_full_items(uint64_t n, const DeviceState& st) {
  const uint64_t round = (uint64_t)std::max(
      1, env_int("DPAR_WIDE_ROUND", st.num_cus));
  const uint64_t r = n % round;
  if (env_int("DPAR_WIDE_TAIL", 1) == 0 || n <= round || 8 * r > 7 * round)
    return n;
  return n - r;
}

struct UnitChoice {
  dpar::Unit unit = dpar::Unit::SEQ;
  int lv_log2t = 0;  // LEVEL: log2 of the chunk capacity in quanta
  int lv_C = 1;      // LEVEL: chunks per block
};

// How work items are evaluated (DPAR_UNIT=seq|level|sub forces one):
//   SEQ   post-order walk, one wavefront per tree: the default;
//   LEVEL the chunk staged in LDS, level by level: when the chunks of a round
//         (per-round executors) or of the whole call number fewer than half
//         a chunk per CU (measured crossover at p = 1152, m = 2^22: 249
//         chunks per round 10.1 ms post-order vs 12.8 ms level; 110 chunks
//         17.9 vs 15.8 ms), or for few short chunks with long chains (a
//         post-order item costs its p/2-load chain however little it
//         carries: p = 1152, m = 4096, b = 205: 117 us post-order, 31 level);
//   WIDE  the post-order walk with kWideQ quanta per lane: a whole call
//         (split, ticket, one fused launch) on 16-byte lanes whose slots
//         fit in LDS (p < 1024) with at least 3/4 of a wide item (16 KB
//         of columns) per CU (7/8 with at most 16 ranks), unless the split
//         up-phase would run post-order items under its residency cap
//         (measured, int32 SUM,
//         split, 192 items: p = 96 107 -> 100 us, p = 288 291 -> 277 us,
//         p = 900 893 -> 881 us; 224 items 5-11% faster; with 160 items
//         post-order items are 0-3% faster; rows of 4 / 8 / 16 MB: p = 36
//         61.4 -> 57.5, 110 -> 103, 211 -> 195 us; p = 128 180 -> 164,
//         340 -> 315, 675 -> 627 us; p = 511 667 -> 611, 1311 -> 1235 us;
//         under the cap, p = 256 .. 768 with 16 MB rows, post-order items
//         are 0-4% faster; 2 wavefronts per item for deeper trees won only
//         at p = 1152 with 4 MB rows and lost up to 30% elsewhere);
//   SUB   eight subtree walks, then the spines: a whole call (split,
//         ticket, one fused launch) in at most two full chunks per CU
//         with p >= 256 (p = 1152, m = 2^16, b = 1: 0.113 vs 0.165 ms;
//         two per CU, p = 1152, m = 2^17: 0.240 vs 0.260 ms), and in
//         place of LEVEL at p >= 256 when the level plan needs more than
//         two items per CU; for launch per round and grid barrier only when
//         a round has half a chunk to two chunks per CU, none of them short
//         (elsewhere it loses).
UnitChoice choose_unit(dpar::Exec ex, const dpar::Schedule& s, int grp,
                       dpar::Path path, dpar::Kind kind, int p,
                       const OpsTable& ops, const DeviceState& st) {
  UnitChoice uc;
  const char* u = std::getenv("DPAR_UNIT");
  const bool forced = u && *u;
  const uint64_t cus = (uint64_t)st.num_cus;
  const bool per_round = ex == dpar::Exec::LAUNCH_PER_ROUND ||
                         ex == dpar::Exec::GRID_BARRIER ||
                         ex == dpar::Exec::ROUNDS ||
                         ex == dpar::Exec::ROUNDS_BARRIER;
  const uint64_t all_items = grouped_units(s, grp);
  const uint64_t items = per_round ? (uint64_t)s.C : all_items;
  const bool whole_call = ex == dpar::Exec::SPLIT ||
                          ex == dpar::Exec::TICKET ||
                          ex == dpar::Exec::DISPATCH;
  const size_t lane_bytes =
      (path == dpar::Path::VEC16 || kind == dpar::Kind::MAT) ? 16 : 4;
  // a one-launch subtree run cuts the columns into whole chunks of 64
  // quanta, whatever the blocks (see allreduce_impl): count those
  const uint64_t sub_items = (s.Q + 63) / 64;
  const bool sub_fits = ops.sub &&
                        dpar::sub_lds_bytes(lane_bytes, ops.sub_ns) <=
                            (size_t)st.lds_limit - dpar::kStaticLdsReserve;
  // Launch per round and grid barrier with rounds of between half a chunk
  // and two chunks per CU: every round is one generation of work items whose
  // chains of p/2 loads set the round's time; subtree items cut the chains.
  // Measured at p = 1152, m = 2^22 fp32, b = 66 (249 chunks per round):
  // launch per round 10.0 -> 7.3 ms, grid barrier 11.5 -> 9.0 ms (the
  // round-structured executor, whose rounds also carry the down-step,
  // 10.0 -> 10.7 ms: not taken there).  With shorter rounds level items
  // win (b = 6532, 3 chunks per round: 143 ms level, 355 ms subtree).
  const bool round_sub = (ex == dpar::Exec::LAUNCH_PER_ROUND ||
                          ex == dpar::Exec::GRID_BARRIER) &&
                         p >= 256 && (uint64_t)s.C >= cus / 2 &&
                         (uint64_t)s.C <= 2 * cus && s.Q >= 32 * all_items;
  // From kSubCrowdRanks ranks on subtree items also take calls of up to
  // four per CU (split; post-order chains of p / 2 loads are then the
  // longer wait): p = 4608, m = 2^18 (1024 items), median of four runs,
  // post-order split 1685 us back to back / 2086 us after a cache flush,
  // subtree split 1528 / 1897 us; at p = 2304 post-order items stay
  // faster (735 / 884 against 798 / 971 us).
  const bool sub_crowd = whole_call && p >= kSubCrowdRanks &&
                         sub_items <= 4 * cus;
  bool want_sub = p >= 256 && sub_fits &&
                  ((whole_call && sub_items <= 2 * cus) || sub_crowd ||
                   round_sub);
  if (ops.lvl) {
    int tmax = -1;
    for (int lg = 6; lg >= 0; --lg) {
      if (dpar::level_lds_bytes(path, kind, p, lg, ops.height + 1) <=
          (size_t)st.lds_limit - dpar::kStaticLdsReserve) {
        tmax = lg;
        break;
      }
    }
    bool want = items < cus / 2 ||
                (p >= 256 && items < 2 * cus && s.Q < 32 * all_items);
    if (forced) want = !std::strcmp(u, "level");
    if (want && tmax >= 0) {
      // largest block (group of grp blocks) in quanta; chunk capacity T =
      // a power of two
      const uint64_t maxq =
          ((s.NL * (uint64_t)grp + s.b - 1) / s.b) * (uint64_t)s.lq;
      // the largest chunk that fits LDS and the block (group)
      int lg_max = 0;
      while (lg_max < tmax && (1ull << lg_max) < maxq) ++lg_max;
      auto chunks = [&](int l) { return (maxq + (1ull << l) - 1) >> l; };
      const uint64_t groups =
          per_round ? 1 : ((uint64_t)s.b + (uint64_t)grp - 1) / (uint64_t)grp;
      // At large p a level item holds only a few quanta of each row; when
      // that takes more than two level items per CU (four from
      // kLvCrowdRanks ranks on) and the subtree item can take the call,
      // it is faster (p = 2304, m = 2^14,
      // b = 1: 1024 level items 0.200 ms, 64 subtree items 0.116 ms;
      // p = 4608: 0.494 vs 0.213 ms; p = 1152 keeps level items: 512 of
      // them, 0.054 vs 0.068 ms; int32 SUM, the rule's b, level items
      // split: p = 2304, m = 4096, 544 level items 67 us, subtree items
      // 91 us; m = 8192, 1088 level items 105 us, subtree 95 us; p = 4608,
      // m = 4096, 1024 level items 149 us, subtree 163 us).
      const uint64_t crowd = p >= kLvCrowdRanks ? 4 : 2;
      const bool crowded = groups * chunks(lg_max) > crowd * cus;
      // Chunk used: the largest whose p * T loads are all in flight at once
      // (1024 threads with kLvBatch loads each), larger only while the items
      // outnumber the CUs.  Measured, int32 SUM, one fused launch: p = 288,
      // m = 875: T = 64 (the largest that fits) 19.4 us, T = 16 14.5 us;
      // m = 25: 15.5 vs 14.2 us; p = 1152, m = 16, b = 13: 19.7 vs
      // 15.3 us; p = 1152, m = 4096: T = 2 (512 items) 41.2 us, T = 4
      // 20.6 us.
      int lg = 0;
      while (lg < lg_max && ((uint64_t)p << (lg + 1)) <= kLvLoadsInFlight)
        ++lg;
      while (lg < lg_max && groups * chunks(lg) > cus) ++lg;
      const int forced_lg = env_int("DPAR_LEVEL_LOG2T", -1);
      if (forced_lg >= 0) lg = std::min(forced_lg, tmax);
      const int lv_C = (int)chunks(lg);
      // A level plan of more than one item per CU ends with a round that
      // is not full, each of its items as long as a whole round's; subtree
      // items, at least a quarter of one per CU, take such a call faster
      // (p = 400, m = 16384: 304 level items 31-33 us, 64 subtree items
      // 27-31 us; m = 24576, p = 350 .. 600: 384 level items 35-49 us,
      // 96 subtree items 28-45 us); with fewer subtree items their chains
      // cost more (p = 1152, m = 8192: 264 level items 43-48 us, 32
      // subtree items 52-55 us).
      const uint64_t lv_items = groups * (uint64_t)lv_C;
      const bool lv_rounds = lv_items > cus && 4 * sub_items >= cus;
      if (forced || !((crowded || lv_rounds) && want_sub)) {
        uc.unit = dpar::Unit::LEVEL;
        uc.lv_log2t = lg;
        uc.lv_C = lv_C;
        return uc;
      }
    }
  }
  if (forced) want_sub = !std::strcmp(u, "sub") && sub_fits;
  if (want_sub) {
    uc.unit = dpar::Unit::SUB;
    return uc;
  }
  const bool wide_fits =
      whole_call && lane_bytes == 16 &&
      dpar::wide_lds_bytes(lane_bytes, ops.height + 1) <=
          (size_t)st.lds_limit - dpar::kStaticLdsReserve;
  const bool seq_capped =
      ex == dpar::Exec::SPLIT && seq_wg_capped(p, all_items, st);
  // With at most kWideLateRanks ranks, post-order items in one fused
  // launch stay faster up to 7/8 of an item per CU (192 items, p = 8 / 12
  // / 16: 16.4 / 20.4 / 24.2 us post-order, 18.2 / 21.0 / 25.8 us wide).
  const uint64_t wide_num = p <= kWideLateRanks ? 7 : 6;
  bool want_wide = wide_fits && !seq_capped &&
                   8 * ((s.Q + dpar::kWideChunk - 1) / dpar::kWideChunk) >=
                       wide_num * cus;
  if (forced) want_wide = !std::strcmp(u, "wide") && wide_fits;
  if (want_wide) uc.unit = dpar::Unit::WIDE;
  return uc;
}

const char* exec_name(dpar::Exec e) {
  switch (e) {
    case dpar::Exec::LAUNCH_PER_ROUND: return "launch_per_round";
    case dpar::Exec::GRID_BARRIER: return "grid_barrier";
    case dpar::Exec::TICKET: return "ticket";
    case dpar::Exec::SPLIT: return "split";
    case dpar::Exec::DISPATCH: return "one_launch_fused";
    case dpar::Exec::TICKET_SPLIT: return "split(ticket up-phase)";
    case dpar::Exec::ROUNDS: return "rounds";
    case dpar::Exec::ROUNDS_BARRIER: return "rounds_barrier";
  }
  return "?";
}

const char* unit_name(dpar::Unit u) {
  return u == dpar::Unit::LEVEL  ? "level"
         : u == dpar::Unit::SUB  ? "subtree"
         : u == dpar::Unit::WIDE ? "wide"
                                 : "postorder";
}

// DPAR_LOG=1: one line per call on stderr with the plan it runs (tree
// height, block count, decomposition, executor, work item), for diagnosis.
void log_plan(int p, size_t m, dpar_dtype_t dtype, dpar_op_t op,
              dpar_alg_t alg, bool rule_b, const dpar::Schedule& s,
              dpar::Path path, dpar::Exec ex, dpar::Unit unit, int waves,
              const dpar::Params& prm, int height) {
  static const char* dts[] = {"int32", "float32", "u32mat2x2"};
  static const char* opn[] = {"sum", "max", "matmul"};
  static const char* algs[] = {"dual_root", "single_tree", "reduce_bcast"};
  const uint64_t items = ((uint64_t)prm.b + (uint64_t)prm.grp - 1) /
                         (uint64_t)prm.grp * (uint64_t)prm.C;
  std::fprintf(stderr,
               "dpar: p=%d m=%zu %s %s alg=%s H=%d b=%d%s lanes=%s "
               "quantum=%d line_quanta=%d tail=%llu exec=%s unit=%s "
               "waves=%d chunks_per_block=%d blocks_per_item=%d items=%llu",
               p, m, dts[(int)dtype], opn[(int)op], algs[(int)alg], height,
               s.b, rule_b ? " (rule)" : "",
               path == dpar::Path::VEC16 ? "16B" : "4B", s.g, s.lq,
               (unsigned long long)s.tail, exec_name(ex), unit_name(unit),
               waves, prm.C, prm.grp, (unsigned long long)items);
  if (unit == dpar::Unit::LEVEL)
    std::fprintf(stderr, " level_chunk_quanta=%d", 1 << prm.lv_log2t);
  if (unit == dpar::Unit::SUB)
    std::fprintf(stderr, " sub_deep=%d", prm.sub_deep);
  if (unit == dpar::Unit::WIDE)
    std::fprintf(stderr, " full_items=%u", prm.wide_full);
  if (ex == dpar::Exec::TICKET) std::fprintf(stderr, " batch=%u", prm.batch);
  std::fprintf(stderr, "\n");
}

// fixed: the allocation-free variant (dual-root trees, AUTO executor, device
// tables in the fixed scratch, no counters).
int allreduce_impl(const void* const* x, void* const* y, int p, size_t m,
                   dpar_dtype_t dtype, dpar_op_t op, int b,
                   const dpar_options_t& opt, hipStream_t stream,
                   bool fixed = false) {
  g_err.clear();
  // the phase event (dpar_set_phase_event) belongs to this call alone,
  // recorded only if it runs the split executor's two passes
  const hipEvent_t phase_event = g_phase_event;
  g_phase_event = nullptr;
  const dpar_exec_t exec = opt.exec;
  const dpar_alg_t alg = opt.alg;
  if (!x || !y) return fail(DPAR_ERR_INVALID_ARG, "null pointer array");
  if (p < 1) return fail(DPAR_ERR_INVALID_ARG, "p must be >= 1");
  if (b < 0) return fail(DPAR_ERR_INVALID_ARG, "b must be >= 0");
  if (!valid_pair(dtype, op))
    return fail(DPAR_ERR_UNSUPPORTED, "unsupported dtype/op pair (%d, %d)",
                (int)dtype, (int)op);
  if (exec < DPAR_EXEC_AUTO || exec > DPAR_EXEC_ROUNDS_BARRIER)
    return fail(DPAR_ERR_INVALID_ARG, "unknown executor %d", (int)exec);
  if (alg < DPAR_ALG_DUAL_ROOT || alg > DPAR_ALG_REDUCE_BCAST)
    return fail(DPAR_ERR_INVALID_ARG, "unknown algorithm %d", (int)alg);
  if (fixed && p > dpar::kFixedMaxRanks)
    return fail(DPAR_ERR_UNSUPPORTED, "p = %d beyond the %d ranks of the "
                "allocation-free entry point", p, dpar::kFixedMaxRanks);
  const bool rounds_exec =
      exec == DPAR_EXEC_ROUNDS || exec == DPAR_EXEC_ROUNDS_BARRIER;
  if (!rounds_exec && (opt.round_begin != 0 || opt.round_end != -1))
    return fail(DPAR_ERR_INVALID_ARG, "a round range needs a ROUNDS executor");
  if (opt.round_begin < 0 || opt.round_end < -1 ||
      (opt.round_end >= 0 && opt.round_end < opt.round_begin))
    return fail(DPAR_ERR_INVALID_ARG, "bad round range [%d, %d)",
                opt.round_begin, opt.round_end);
  // every output row starts on a 128-byte cache line (else the broadcast
  // pass aligns each row's stores itself)
  // one branch-free pass (OR of all addresses, any null); only a call that
  // fails a check walks the ranks again to name the first offender
  uintptr_t or_x = 0, or_y = 0;
  bool any_null = false;
  for (int i = 0; i < p; ++i) {
    const uintptr_t a = (uintptr_t)x[i], c = (uintptr_t)y[i];
    or_x |= a;
    or_y |= c;
    any_null |= (a == 0) | (c == 0);
  }
  if (any_null || ((or_x | or_y) & 3) || ((or_x | or_y) >> 48)) {
    for (int i = 0; i < p; ++i) {
      if (!x[i] || !y[i])
        return fail(DPAR_ERR_INVALID_ARG, "null buffer for rank %d", i);
      const uintptr_t a = (uintptr_t)x[i], c = (uintptr_t)y[i];
      if ((a | c) & 3)
        return fail(DPAR_ERR_INVALID_ARG,
                    "rank %d buffer not 4-byte aligned", i);
      if (((a | c) >> 48) != 0)
        return fail(DPAR_ERR_UNSUPPORTED, "rank %d address above 2^48", i);
    }
  }
  const bool rows_lines = (or_y & 127) == 0;
  const bool xrows_lines = (or_x & 127) == 0;  // every input row on a line
  if (m == 0) return DPAR_SUCCESS;
  const bool rule_b = b == 0;
  if (b == 0) b = (int)dpar::block_rule(p, m, 0.0, 0.0);
  if ((size_t)b > m)
    return fail(DPAR_ERR_INVALID_ARG, "b = %d exceeds m = %zu", b, m);
  const size_t esz = elem_size(dtype);
  if (m > (size_t)1 << 40)
    return fail(DPAR_ERR_UNSUPPORTED, "m beyond 2^40 elements");

  int r0 = 0, r1 = 0;
  if (rounds_exec) {
    const int R = dpar_schedule_rounds(p, b, alg);
    if (R < 0) return R;
    r0 = opt.round_begin;
    r1 = opt.round_end < 0 ? R : opt.round_end;
    if (r1 > R)
      return fail(DPAR_ERR_INVALID_ARG, "round range [%d, %d) beyond R = %d",
                  r0, r1, R);
  }
  // One element per lane when 4-element quanta would leave trailing
  // elements and either the round-structured executors run (they have no
  // separate pass for them) or the call is small enough that the launch
  // that pass needs costs more than the wider lanes save (DPAR_SCALAR=1:
  // always).
  const bool one_per_lane = one_element_per_lane(p, m, dtype, rounds_exec);
  dpar::Schedule s;
  dpar::Path path;
  choose_schedule(m, dtype, b, one_per_lane, &s, &path);
  if ((unsigned __int128)s.NL * (unsigned)(b + 1) >= ((unsigned __int128)1 << 63))
    return fail(DPAR_ERR_UNSUPPORTED, "m * b beyond the index range");
  {
    // work items = b * chunks per block, counted before the int narrowing
    const uint64_t max_lines = (s.NL + (uint64_t)b - 1) / (uint64_t)b;
    const uint64_t per_chunk = 64 / (uint64_t)s.lq;
    const uint64_t c64 = (max_lines + per_chunk - 1) / per_chunk;
    if ((unsigned __int128)c64 * (unsigned)b >= ((unsigned __int128)1 << 31))
      return fail(DPAR_ERR_UNSUPPORTED, "more than 2^31 work items");
  }

  std::lock_guard<std::mutex> lock(g_mu);
  // aliasing rules: checked before any device work; a pointer set that
  // passed for this row length is not sorted again
  if (!alias_cached(x, y, p, m * esz)) {
    if (!aliasing_ok(x, y, p, m * esz))
      return fail(DPAR_ERR_ALIAS, "output buffers overlap each other or "
                                  "partially overlap an input");
    alias_remember(x, y, p, m * esz);
  }
  if (rounds_exec && r0 == r1) return DPAR_SUCCESS;
  // One rank: the reduction is x_0 itself and the delivery a copy into y_0
  // (nothing in place).  The round-structured executors keep their rounds.
  if (p == 1 && !rounds_exec) {
    if (env_int("DPAR_LOG", 0) != 0)
      std::fprintf(stderr, "dpar: p=1 m=%zu exec=copy\n", m);
    if (x[0] == y[0]) return DPAR_SUCCESS;
    const hipError_t e = dpar::copy_row((uint64_t)(uintptr_t)x[0],
                                        (uint64_t)(uintptr_t)y[0], m * esz,
                                        stream);
    return e == hipSuccess ? DPAR_SUCCESS : hip_fail(e, "copy launch");
  }
  // Under stream capture (a HIP graph being recorded) a call may only
  // enqueue kernels: the device tables and the staged pointer set must exist
  // already (an eager call with the same arguments made them), the staging
  // slot is pinned for the graph's lifetime, and no event is recorded.
  hipStreamCaptureStatus cap = hipStreamCaptureStatusNone;
  {
    hipError_t e = hipStreamIsCapturing(stream, &cap);
    if (e != hipSuccess) return hip_fail(e, "hipStreamIsCapturing");
  }
  const bool capturing = cap != hipStreamCaptureStatusNone;
  if (capturing && fixed)
    return fail(DPAR_ERR_UNSUPPORTED, "the allocation-free entry point "
                "cannot be captured into a graph");
  if (capturing && (exec == DPAR_EXEC_GRID_BARRIER ||
                    exec == DPAR_EXEC_ROUNDS_BARRIER))
    return fail(DPAR_ERR_UNSUPPORTED,
                "the cooperative executors cannot be captured into a graph");
  const bool single = alg != DPAR_ALG_DUAL_ROOT;
  if (capturing) {
    int dev = 0;
    hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
    auto it = g_devices.find(dev);
    if (it == g_devices.end() ||
        !it->second->ops.count(std::make_pair(p, single ? 1 : 0)))
      return fail(DPAR_ERR_UNSUPPORTED,
                  "capture: make one eager call with these arguments first");
  }
  DeviceState* st = nullptr;
  FixedState* fx = nullptr;
  const OpsTable* ops = nullptr;
  int rc = DPAR_SUCCESS;
  if (fixed) {
    rc = get_fixed(&fx);
    if (rc) return rc;
    st = &fx->info;
    rc = fixed_tables(fx, p, stream, &ops);
  } else {
    rc = get_state(&st);
    if (rc) return rc;
    rc = get_ops(st, p, single, &ops);
  }
  if (rc) return rc;
  if (rounds_exec && !ops->dn)
    return fail(DPAR_ERR_UNSUPPORTED, "ROUNDS executors need p < 2^24");

  int waves = chunk_waves(p);
  const int nslots = ops->height + 1;
  const dpar::Kind kind = kind_of(dtype, op);
  if (dpar::lds_bytes(path, kind, waves, nslots) > 65536 && waves == 2)
    waves = 1;
  if (dpar::lds_bytes(path, kind, waves, nslots) > 65536)
    return fail(DPAR_ERR_UNSUPPORTED, "tree too deep for the LDS slots");

  StageSlot* slot = nullptr;
  const uint64_t* ptr_dev = nullptr;
  if (fixed) {
    rc = fixed_pointers(fx, x, y, p, stream, &ptr_dev);
    if (rc) return rc;
  } else {
    if (!find_staged(st, x, y, p, &slot)) {
      if (capturing)
        return fail(DPAR_ERR_UNSUPPORTED, "capture: make one eager call with "
                                          "these pointer arrays first");
      rc = stage_pointers(st, x, y, p, stream, &slot);
      if (rc) return rc;
    }
    rc = order_after_copy(slot, stream, capturing);
    if (rc) return rc;
    if (capturing) slot->pinned = true;
    ptr_dev = slot->dev;
  }

  // ticket and barrier words (none for the allocation-free variant, whose
  // executors use none)
  unsigned* slot_base = nullptr;
  unsigned* line = nullptr;
  if (!fixed) {
    const unsigned cslot = st->next_counter++ % kCounterSlots;
    slot_base = st->counters + (size_t)cslot * kLinesPerSlot * kCounterStride;
    line = slot_base + (size_t)2 * dpar::kTicketCounters * kCounterStride;
  }
  dpar::Params prm{};
  prm.p = p;
  prm.n_a = ops->n_a;
  prm.nslots = nslots;
  prm.dual = p >= 2;
  prm.Q = s.Q;
  prm.NL = s.NL;
  prm.lq = (uint32_t)s.lq;
  prm.qbase = 0;
  prm.b = s.b;
  prm.C = s.C;
  dpar::Exec ex = device_exec(exec, p, 2ull * p * m * esz);
  prm.grp = block_group(ex, s);
  {
    // Work items per ticket: a claim is an atomic at device scope, whose
    // round trip costs about as much as a short work item, so items of few
    // ranks are claimed several at a time (about kTicketRankLoads rank loads
    // per claim), leaving at least two batches per CU (measured, ticket
    // executor, b = 1: p = 36, m = 2^20 int32 0.224 / 0.144 / 0.103 /
    // 0.140 ms with 1 / 2 / 8 / 16 items per claim; p = 64, m = 2^18
    // matrices 0.283 / 0.208 / 0.179 / 0.195 ms; p = 1152, m = 2^16 one item
    // 0.120 ms, two 0.156 ms).
    const uint64_t units = grouped_units(s, prm.grp);
    uint64_t k = (kTicketRankLoads + (uint64_t)p - 1) / (uint64_t)p;
    const uint64_t fair = units / (2ull * (uint64_t)st->num_cus);
    if (k > fair) k = fair;
    if (k < 1) k = 1;
    prm.batch = (unsigned)env_int("DPAR_TICKET_BATCH", (int)k);
    if (prm.batch < 1) prm.batch = 1;
  }
  prm.ticket = slot_base;
  prm.done = fixed ? nullptr
                   : slot_base + (size_t)dpar::kTicketCounters * kCounterStride;
  prm.bar_count = fixed ? nullptr : line + 0;
  prm.bar_gen = fixed ? nullptr : line + 1;
  prm.bar_quit = fixed ? nullptr : line + 2;
  prm.err = fixed ? nullptr
                  : st->counters + (size_t)kCounterSlots * kLinesPerSlot *
                                       kCounterStride;
  prm.spin_limit = spin_limit();

  dpar::Tables tab;
  tab.xp = ptr_dev;
  tab.yp = ptr_dev + p;
  tab.ops = ops->dev;
  tab.lvl = ops->lvl;
  tab.dn = ops->dn;
  tab.dord = ops->dord;
  tab.doff_host = ops->doff.empty() ? nullptr : ops->doff.data();

  // outputs the non-fused up-step writes: y_0 for the split executor (the
  // broadcast pass copies it on), the real root(s) for the round structure
  prm.out0 = 0;
  prm.out1 = -1;
  if (rounds_exec) {
    prm.out0 = ops->root_a;
    prm.out1 = ops->root_b;
  }
  prm.dshift = alg == DPAR_ALG_REDUCE_BCAST ? b - 1 : 0;
  prm.dheight = ops->real_height;
  prm.r0 = r0;
  prm.r1 = r1;

  const UnitChoice uc = choose_unit(ex, s, prm.grp, path, kind, p, *ops, *st);
  // AUTO: a call that runs in subtree work items (at most two per CU) runs
  // them as one fused launch rather than split: each item's y goes from
  // registers to all p outputs while the few other items still read, and
  // the broadcast pass's many short workgroups (and their launch) are gone.
  // Measured, int32 SUM, cold caches, the sqrt(m log2 p) rule's b: p = 1152,
  // m = 2^16 (256 items) split 0.126 ms, fused 0.107 ms; p = 2304,
  // m = 57344 (224 items) 0.199 vs 0.180 ms; p = 576, m = 57344 0.063 vs
  // 0.057 ms; p = 288, m = 115712 (452 items) 0.060 vs 0.055 ms; down to a
  // quarter of an item per CU in back-to-back calls (64 items, m = 16384:
  // p = 700 46.0 -> 41.9 us, p = 1152 58.5 -> 51.0 us, p = 2304 102.0 ->
  // 93.7 us, p = 4608 185.9 -> 175.2 us; after a cache flush within 2%
  // either way); with fewer the chains dominate and fused is no better
  // (p = 2304, m = 14336, 56 items: 0.107 vs 0.117 ms).  Calls that take
  // post-order items on long rows stay split, which is faster there from
  // 256 MB up (p = 36 .. 2304: 8-35% at 1-38 GB).
  // Beyond two items per CU (many ranks, above) split stays faster in both
  // regimes (p = 4608, m = 2^18: fused 1857 / 1722 us, split 1528 /
  // 1897 us back to back / after a flush; the fused launch's p writes per
  // item then overlap the reads of the items after it).
  if (exec == DPAR_EXEC_AUTO && ex == dpar::Exec::SPLIT &&
      uc.unit == dpar::Unit::SUB &&
      4 * ((s.Q + 63) / 64) >= (uint64_t)st->num_cus &&
      (s.Q + 63) / 64 <= 2 * (uint64_t)st->num_cus)
    ex = dpar::Exec::DISPATCH;
  // AUTO, wide items: with at most one per CU they all run at once, read
  // their rows together and then write y together, so one fused launch
  // keeps reads and writes apart in time and saves the broadcast pass; the
  // p writes per item then cost less than that pass as long as p is small.
  // Measured, int32 SUM, m = 2^20 (256 items), cold caches, split -> fused
  // (best of 3 runs): p = 8 24.5 -> 18.2 us, p = 24 43.1 -> 37.8 us,
  // p = 36 57.8 -> 56.5 us (on another box 2-3% the other way, and on a
  // third within 2%); p = 32, 40 and 48 were 1-5% slower fused on that
  // third box, p = 64 89.3 -> 91.7 us; with two items per CU (p = 36,
  // m = 2^21) 103 -> 109 us.  With up to 20 ranks (two or three items fit
  // per CU by LDS) the fused launch also wins with up to two items per CU,
  // when it runs full items only (split -> fused, full items only / with
  // tail items: p = 12, 401 items 1.00 -> 0.84 / 0.96; p = 16, 448 items
  // 1.00 -> 0.95 / 1.07; p = 20, 480 items 1.00 -> 0.93 / 1.05; p = 24,
  // 0.95-1.08, taken split).  With very few ranks the split executor's
  // extra traffic (y_0 written, then read back: 1/p of the call's bytes)
  // outweighs the interleaving at any size: p = 2, m = 2^22 (1024 items)
  // 35.6 -> 17.6 us; p = 8, 1024 / 2048 / 4096 items 59.4 -> 51.6,
  // 106.8 -> 102.0, 204.5 -> 202.3 us; 256 to 640 items 8-19% faster.
  const uint64_t wide_n = (s.Q + dpar::kWideChunk - 1) / dpar::kWideChunk;
  const uint64_t ncu = (uint64_t)st->num_cus;
  const bool wide_fuse_two =
      p <= kWideFuseTwoRanks && wide_n > ncu && wide_n <= 2 * ncu;
  if (exec == DPAR_EXEC_AUTO && ex == dpar::Exec::SPLIT &&
      uc.unit == dpar::Unit::WIDE &&
      (p <= kWideFuseAnyRanks || wide_fuse_two ||
       (p <= kWideFuseMaxRanks && wide_n <= ncu)))
    ex = dpar::Exec::DISPATCH;
  // AUTO, post-order items on short rows: one fused launch saves the split
  // executor's second launch, the y_0 round trip and the broadcast pass's
  // fill and drain, which on rows of at most seq_fuse_row_bytes(p) cost
  // more than reading and writing in the same launch.  Measured, int32 SUM,
  // cold caches, split -> fused: p = 36, m = 2^19 (2 MB rows) 36.2 ->
  // 31.9 us; 2.5 MB rows: p = 12 24.2 -> 18.9 us, p = 24 32.6 -> 26.7 us,
  // p = 48 52.7 -> 51.0 us; 3 MB rows: p = 8 / 12 / 16 20.9 / 25.7 / 28.5
  // -> 16.4 / 20.4 / 24.2 us; p = 64, m = 393216 (1.5 MB rows) 45.7 ->
  // 42.7 us; 1 MB rows: p = 128 60.4 -> 53.4 us, p = 288 120.6 ->
  // 110.7 us, p = 511 201.7 -> 189.2 us, p = 700 to 2304 within 2% either
  // way, p = 4608 2093 -> 1861 us.  Those calls follow a 512 MB write that
  // flushes the caches; in back-to-back calls (also on two alternating sets
  // of buffers, so not from reused data; after a 32 MB write too) the split
  // executor is faster: fused on 1 MB rows
  // is then 9-16% slower from p = 128 on (p = 1152: 388 vs 464 us; at
  // p = 96 as fast), on 512 KB rows 3-7% slower from p = 400 on and
  // faster up to p = 200 (44.4 vs 47.8 us), so beyond 96 ranks only rows
  // of up to 512 KB are fused (cold, p = 400 .. 1152: 12-16% faster).  One
  // step longer the split executor wins (p = 64, 2 MB rows: 58.6 vs 62.0 us;
  // p = 128, 1.5 MB rows: 80.2 vs 85.1 us).
  if (exec == DPAR_EXEC_AUTO && ex == dpar::Exec::SPLIT &&
      uc.unit == dpar::Unit::SEQ &&
      (uint64_t)m * esz <= seq_fuse_row_bytes(p))
    ex = dpar::Exec::DISPATCH;
  // AUTO, level items: a fused level item writes its chunk (a few quanta)
  // to each of the p outputs, piece by piece; with many ranks the
  // broadcast pass's whole tiles are faster, with few ranks the fused
  // launch (int32 SUM, the rule's b, fused -> split, after a cache flush:
  // p = 400, m = 16384 33.2 -> 35.2 us; p = 511 24.0 -> 28.6 us; p = 1152,
  // m = 8192 57.3 -> 48.2 us; p = 2304, m = 1024 36.6 -> 33.4 us;
  // p = 4608, m = 1024 73.9 -> 53.4 us; p = 1152, m = 1024 and 4096 2-4%
  // slower split, but in back-to-back calls 24.7 -> 18.7 us and 31.7 ->
  // 30.1 us; from 512 ranks on with at least one item per CU: p = 700,
  // m = 8192 38.9 -> 34.3 us back to back, 38.8 -> 35.8 us after a flush;
  // p = 900 42.9 -> 37.2 us).
  if (exec == DPAR_EXEC_AUTO && uc.unit == dpar::Unit::LEVEL &&
      (ex == dpar::Exec::SPLIT || ex == dpar::Exec::DISPATCH)) {
    const uint64_t lv_items =
        grouped_units(s, prm.grp) / (uint64_t)s.C * (uint64_t)uc.lv_C;
    const bool split = p >= kLvSplitRanks ||
                       (p >= kLvSplitManyRanks &&
                        lv_items >= (uint64_t)st->num_cus);
    ex = split ? dpar::Exec::SPLIT : dpar::Exec::DISPATCH;
  }
  const dpar::Unit unit = uc.unit;
  prm.nlev = ops->height + 1;
  if (unit == dpar::Unit::LEVEL) {
    prm.C = uc.lv_C;
    prm.lv_log2t = uc.lv_log2t;
    prm.batch = 1;
    if (grouped_units(s, prm.grp) / (uint64_t)s.C * (uint64_t)prm.C >=
        (1ull << 31))
      return fail(DPAR_ERR_UNSUPPORTED, "more than 2^31 work items");
  }
  if (unit == dpar::Unit::SUB) {
    tab.lvl = ops->sub;
    prm.nslots = ops->sub_ns;
    // One launch of subtree work items has fewer than two per CU, all
    // resident at once, so its items need not follow the blocks: the
    // columns are cut into whole chunks of 64 quanta, as with b = 1 (at
    // p = 1152, m = 2^16, b = 817: 256 items instead of 273 groups of three
    // blocks, 0.079 -> 0.063 ms for the up-phase).  Element-wise, so the
    // result does not depend on the cut.
    if (ex == dpar::Exec::SPLIT || ex == dpar::Exec::DISPATCH ||
        ex == dpar::Exec::TICKET) {
      const dpar::Schedule s1 = dpar::make_schedule(m, 1, s.g, 8);
      prm.b = 1;
      prm.NL = s1.NL;
      prm.lq = (uint32_t)s1.lq;
      prm.C = s1.C;
      prm.grp = 1;
    }
    // Long parts and at most one item per CU: a deeper load pipeline per
    // wavefront shortens the chains (its registers leave room for one
    // subtree workgroup per CU instead of two).  Measured, int32 SUM, split:
    // p = 2304, m = 2^14: 0.112 -> 0.101 ms; p = 4608, m = 2^14: 0.210 ->
    // 0.188 ms; p = 1152, m = 2^14, b = 207: 0.064 -> 0.060 ms; with 384
    // items at p = 1152 (residency halved) 5% slower, at p <= 576 1-3%.
    const uint64_t sub_items =
        ((uint64_t)prm.b + (uint64_t)prm.grp - 1) / (uint64_t)prm.grp *
        (uint64_t)prm.C;
    prm.sub_deep = env_int("DPAR_SUB_DEEP",
                           p >= kSubDeepMinRanks &&
                               sub_items <= (uint64_t)st->num_cus);
  }
  if (unit == dpar::Unit::WIDE) {
    // One launch of wide items (one-launch executors only): item t takes the
    // quanta [t kWideChunk, (t + 1) kWideChunk), whatever the blocks, as the
    // subtree items above (element-wise, so the result does not depend on
    // the cut); each item is claimed on its own.
    const dpar::Schedule s1 = dpar::make_schedule(m, 1, s.g, 8);
    prm.b = 1;
    prm.NL = s1.NL;
    prm.lq = (uint32_t)s1.lq;
    prm.grp = 1;
    prm.batch = 1;
    const uint64_t n = (s.Q + dpar::kWideChunk - 1) / dpar::kWideChunk;
    // a fused launch of at most two items per CU with few ranks: full items
    // only (see the executor choice above), unless DPAR_WIDE_ROUND sets the
    // rounds
    const bool full_only = ex == dpar::Exec::DISPATCH &&
                           p <= kWideFuseTwoRanks &&
                           n <= 2 * (uint64_t)st->num_cus &&
                           !std::getenv("DPAR_WIDE_ROUND");
    const uint64_t full = full_only ? n : wide_full_items(n, *st);
    prm.wide_full = (uint32_t)full;
    prm.C = (int)(full + (s.Q - std::min(s.Q, full * dpar::kWideChunk) +
                          dpar::kWideTailChunk - 1) /
                             dpar::kWideTailChunk);
  }
  // round-structured down-step: two ranks per wavefront per work item, the
  // largest block in pieces of kDownPiece quanta
  prm.dslice = 2 * (unit == dpar::Unit::LEVEL ? 16
                    : unit == dpar::Unit::SUB ? dpar::kSubParts
                                              : waves);
  {
    const uint64_t maxq = ((s.NL + s.b - 1) / s.b) * (uint64_t)s.lq;
    const uint64_t np = (maxq + dpar::kDownPiece - 1) / dpar::kDownPiece;
    const uint64_t slices = ((uint64_t)p + prm.dslice - 1) / prm.dslice;
    if (rounds_exec && (uint64_t)prm.C + slices * np >= (1ull << 31))
      return fail(DPAR_ERR_UNSUPPORTED, "more than 2^31 work items per round");
    prm.npieces = (int)std::max<uint64_t>(np, 1);
  }

  // the up-phase of the split executor: one workgroup per work item handed
  // out by the hardware in round order (persistent ticketed workgroups on
  // request, for comparison)
  dpar::Exec up = ex;
  if (ex == dpar::Exec::SPLIT && !fixed) {
    const char* v = std::getenv("DPAR_SPLIT_UP");
    if (v && !std::strcmp(v, "ticket")) up = dpar::Exec::TICKET_SPLIT;
  }
  // The split executor's up-phase reads a chunk of every one of the p rows
  // per work item.  With long walks and many work items it reads HBM faster
  // with fewer workgroups resident per CU (fewer rows streamed at once) than
  // with a full CU; the cap is set through the LDS each workgroup requests.
  size_t lds_floor = 0;
  const char* cap_env = std::getenv("DPAR_SEQ_WG_PER_CU");
  const bool cap_forced = cap_env && *cap_env;
  if (up == dpar::Exec::SPLIT && unit == dpar::Unit::SEQ &&
      (cap_forced || seq_wg_capped(p, grouped_units(s, prm.grp), *st))) {
    const int per_cu = env_int("DPAR_SEQ_WG_PER_CU", kSeqWgPerCu);
    if (per_cu > 0)
      lds_floor = (size_t)st->lds_per_cu / (size_t)(per_cu + 1) + 1024;
    if (lds_floor > (size_t)st->lds_limit) lds_floor = 0;
  }
  // the split up-phase on input rows off the 128-byte lines: each XCD takes
  // a contiguous run of work items (plan.hpp xcd_run_index; rows 16 bytes
  // past a line, p = 1152: m = 2^22 up-phase 3.25 -> 3.07 ms, m = 2^18
  // 227 -> 186 us)
  if (up == dpar::Exec::SPLIT && path == dpar::Path::VEC16 && !xrows_lines)
    prm.xcd_runs = 1;
  if (up == dpar::Exec::SPLIT)
    prm.xcd_runs = env_int("DPAR_XCD_RUNS", prm.xcd_runs) != 0;
  if (env_int("DPAR_LOG", 0) != 0)
    log_plan(p, m, dtype, op, alg, rule_b, s, path, up, unit, waves, prm,
             ops->real_height);
  // The cooperative executors start from zeroed barrier words (arrivals,
  // generation, give-up): a call whose wait gave up may leave them out of
  // step, and its counter slot comes round again kCounterSlots calls later.
  // (These executors are refused under capture, so no graph records this.)
  if (ex == dpar::Exec::GRID_BARRIER || ex == dpar::Exec::ROUNDS_BARRIER) {
    const hipError_t ez =
        hipMemsetAsync(line, 0, kCounterStride * sizeof(unsigned), stream);
    if (ez != hipSuccess) return hip_fail(ez, "hipMemsetAsync barrier words");
  }
  hipError_t e = dpar::launch(kind, path, unit, waves, up, tab, prm, stream,
                              st->num_cus, lds_floor);
  if (e != hipSuccess) return hip_fail(e, "kernel launch");
  if (s.tail > 0) {
    // the elements after the last whole 16-byte quantum: one more chunk of
    // the last block, with one scalar per lane
    dpar::Params tp = prm;
    tp.nslots = nslots;  // the post-order item's slots (SUB changed prm's)
    tp.Q = s.tail;
    tp.NL = s.tail;
    tp.lq = 1;
    tp.qbase = s.Q * (uint64_t)s.g;
    tp.b = 1;
    tp.C = 1;
    tp.grp = 1;
    tp.batch = 1;
    tp.xcd_runs = 0;
    // at most 3 elements: evaluated level by level (all p loads at once)
    // where the level table exists; a post-order walk would be a chain of
    // p / 2 dependent loads (p = 288, 2125 elements: 47 us per call with
    // the walk)
    dpar::Tables tt = tab;
    tt.lvl = ops->lvl;
    tp.lv_log2t = 2;
    const bool level =
        p >= 2 && ops->lvl &&
        dpar::level_lds_bytes(dpar::Path::SCALAR, kind, p, tp.lv_log2t,
                              tp.nlev) <=
            (size_t)st->lds_limit - dpar::kStaticLdsReserve;
    e = dpar::launch(kind, dpar::Path::SCALAR,
                     level ? dpar::Unit::LEVEL : dpar::Unit::SEQ, waves,
                     dpar::Exec::LAUNCH_PER_ROUND, tt, tp, stream,
                     st->num_cus, 0);
    if (e != hipSuccess) return hip_fail(e, "tail launch");
  }
  if (ex == dpar::Exec::SPLIT) {
    if (phase_event) {
      e = hipEventRecord(phase_event, stream);
      if (e != hipSuccess) return hip_fail(e, "hipEventRecord phase event");
    }
    // y_0 now holds y for the whole chunked part; stream it to y_1..y_{p-1}
    const uint64_t main_bytes = s.Q * (uint64_t)s.g * esz;
    int span_kb = env_int("DPAR_BCAST_SPAN_KB", kBcastSpanKB);
    if (span_kb <= 0) span_kb = kBcastSpanKB;
    const uint64_t span = (uint64_t)span_kb << 10;
    // passes that write at most kBcastFastDivMaxBytes: each workgroup finds
    // its row and tile by multiplication rather than 64-bit division
    const bool fastdiv =
        env_int("DPAR_BCAST_FASTDIV",
                main_bytes * (uint64_t)(p - 1) <= kBcastFastDivMaxBytes) != 0;
    e = dpar::broadcast(tab, p, main_bytes, path == dpar::Path::VEC16,
                        rows_lines, span, fastdiv, stream);
    if (e != hipSuccess) return hip_fail(e, "broadcast launch");
  }
  return DPAR_SUCCESS;
}

}  // namespace

extern "C" {

int dpar_allreduce_ex(const void* const* x, void* const* y, int p, size_t m,
                      dpar_dtype_t dtype, dpar_op_t op, int b,
                      dpar_exec_t exec, hipStream_t stream) {
  const dpar_options_t opt{DPAR_ALG_DUAL_ROOT, exec, 0, -1};
  return allreduce_impl(x, y, p, m, dtype, op, b, opt, stream);
}

int dpar_allreduce_opt(const void* const* x, void* const* y, int p, size_t m,
                       dpar_dtype_t dtype, dpar_op_t op, int b,
                       const dpar_options_t* opt, hipStream_t stream) {
  const dpar_options_t dflt{DPAR_ALG_DUAL_ROOT, DPAR_EXEC_AUTO, 0, -1};
  return allreduce_impl(x, y, p, m, dtype, op, b, opt ? *opt : dflt, stream);
}

int dpar_allreduce(const void* const* x, void* const* y, int p, size_t m,
                   dpar_dtype_t dtype, dpar_op_t op, int b,
                   hipStream_t stream) {
  return dpar_allreduce_ex(x, y, p, m, dtype, op, b, DPAR_EXEC_AUTO, stream);
}

int dpar_allreduce_noalloc(const void* const* x, void* const* y, int p,
                           size_t m, dpar_dtype_t dtype, dpar_op_t op, int b,
                           hipStream_t stream) {
  const dpar_options_t opt{DPAR_ALG_DUAL_ROOT, DPAR_EXEC_AUTO, 0, -1};
  return allreduce_impl(x, y, p, m, dtype, op, b, opt, stream, true);
}

int dpar_check_status(hipStream_t stream) {
  g_err.clear();
  hipError_t e = hipStreamSynchronize(stream);
  if (e != hipSuccess) return hip_fail(e, "hipStreamSynchronize");
  std::lock_guard<std::mutex> lock(g_mu);
  DeviceState* st = nullptr;
  int rc = get_state(&st);
  if (rc) return rc;
  unsigned* errw = st->counters + (size_t)kCounterSlots * kLinesPerSlot *
                                      kCounterStride;
  unsigned flag = 0;
  e = hipMemcpy(&flag, errw, sizeof flag, hipMemcpyDeviceToHost);
  if (e != hipSuccess) return hip_fail(e, "hipMemcpy status");
  if (flag) {
    // a barrier wait gave up: report it once (each call zeroes its own
    // barrier words, so only the report word is cleared here)
    e = hipMemset(errw, 0, sizeof(unsigned));
    if (e != hipSuccess) return hip_fail(e, "hipMemset");
    return fail(DPAR_ERR_TIMEOUT,
                "a grid-barrier wait exceeded its spin limit: a GRID_BARRIER "
                "call's outputs are complete (its rounds ran unordered), a "
                "ROUNDS_BARRIER call's outputs are undefined");
  }
  return DPAR_SUCCESS;
}

int dpar_finalize(void) {
  g_err.clear();
  std::lock_guard<std::mutex> lock(g_mu);
  int prev = -1;
  (void)hipGetDevice(&prev);
  for (auto& kv : g_devices) {
    DeviceState* st = kv.second.get();
    (void)hipSetDevice(st->device);
    (void)hipDeviceSynchronize();
    for (auto& o : st->ops) free_ops(o.second);
    for (auto& s : st->stage) {
      if (s.ev) (void)hipEventDestroy(s.ev);
      if (s.host) (void)hipHostFree(s.host);
      if (s.dev) (void)hipFree(s.dev);
    }
    for (const TableBuf& t : st->free_tables) (void)hipFree(t.dev);
    for (const TableBuf& t : st->retired_tables) (void)hipFree(t.dev);
    if (st->counters) (void)hipFree(st->counters);
  }
  g_devices.clear();
  g_alias_ok.clear();
  // the fixed scratch stays (it lives as long as the process); only the
  // record of what it holds is dropped
  for (FixedState& f : g_fixed) {
    f.tables_p = 0;
    f.ptr_key.clear();
  }
  if (prev >= 0) (void)hipSetDevice(prev);
  return DPAR_SUCCESS;
}

}  // extern "C"
