// Happens-before checker for the stage executor (test infrastructure).
//
// The stage library's host code (stage.cpp, planner.cpp, errors.cpp) is
// compiled for the CPU against the stand-in HIP headers in fakeinc/; every
// stream operation it issues lands here.  Streams carry vector clocks:
// an operation on stream S advances S's own component; recording an event
// snapshots S's clock into it; waiting on an event joins the event's clock
// into S's; a host synchronisation joins a stream's clock into the host's,
// and every operation enqueued afterwards starts from the host's clock.
// Every kernel launch and copy declares the byte ranges it reads and writes
// (hb_kernels.cpp); the shadow memory keeps, per byte range, the last write
// and the last read of each stream, and reports a race when an access is not
// ordered after a conflicting earlier one:
//   - a read not ordered after the last write of its bytes,
//   - a write not ordered after the last write or any read since it.
// That covers the executor's rules: every read of a tensor follows its
// producer, every reuse of a slot follows the last read of its previous
// contents, and every host-to-device copy completes before its consumer.
#include <algorithm>
#include <cstdint>
#include <cstdio>
#include <cstring>
#include <map>
#include <string>
#include <vector>

#include "hb.h"
#include "hip/hip_ext.h"
#include "hip/hip_runtime.h"

struct HbStream {
  int id;
  std::string name;
};
struct HbEvent {
  std::vector<uint64_t> vc;
  bool recorded = false;
};

namespace {

struct Acc {
  int stream = -1;   // -1: none
  uint64_t clk = 0;
  uint64_t op = 0;
};

struct Seg {
  uint64_t end;
  Acc w;
  std::vector<Acc> r;   // latest read per stream since the last write
};

struct OpInfo {
  std::string name;
  int stream;
};

struct State {
  std::vector<HbStream*> streams;              // id 0: host
  std::vector<std::vector<uint64_t>> vc;       // per stream id
  std::map<uint64_t, Seg> shadow;
  std::vector<OpInfo> ops;                     // op id -> info (index 0 unused)
  std::vector<std::string> races;
  std::map<uint64_t, std::pair<uint64_t, std::string>> regions;   // start -> (end, name)
  int64_t waits = 0, drop_wait = -1;
  HbStream* null_stream = nullptr;
  State() {
    streams.push_back(new HbStream{0, "host"});
    vc.push_back(std::vector<uint64_t>(1, 0));
    ops.push_back({"", 0});
  }
};

State& S() {
  static State s;
  return s;
}

void join(std::vector<uint64_t>& a, const std::vector<uint64_t>& b) {
  if (a.size() < b.size()) a.resize(b.size(), 0);
  for (size_t i = 0; i < b.size(); ++i) a[i] = std::max(a[i], b[i]);
}

uint64_t comp(const std::vector<uint64_t>& v, int i) { return (size_t)i < v.size() ? v[i] : 0; }

HbStream* resolve(hipStream_t s) {
  if (s) return s;
  State& st = S();
  if (!st.null_stream) st.null_stream = static_cast<HbStream*>(hb_new_stream("null"));
  return st.null_stream;
}

std::string where(uint64_t a) {
  State& st = S();
  auto it = st.regions.upper_bound(a);
  if (it != st.regions.begin()) {
    --it;
    if (a < it->second.first) {
      char buf[64];
      snprintf(buf, sizeof(buf), "+0x%llx", (unsigned long long)(a - it->first));
      return it->second.second + buf;
    }
  }
  char buf[32];
  snprintf(buf, sizeof(buf), "0x%llx", (unsigned long long)a);
  return buf;
}

// Split so that a segment boundary falls at x (if x lies inside a segment).
void split_at(uint64_t x) {
  auto& m = S().shadow;
  auto it = m.upper_bound(x);
  if (it == m.begin()) return;
  --it;
  if (it->first < x && x < it->second.end) {
    Seg right = it->second;
    it->second.end = x;
    m.emplace(x, right);
  }
}

// Segments exactly covering [a, b), created empty where nothing was touched.
std::vector<std::map<uint64_t, Seg>::iterator> cover(uint64_t a, uint64_t b) {
  auto& m = S().shadow;
  split_at(a);
  split_at(b);
  std::vector<std::map<uint64_t, Seg>::iterator> out;
  uint64_t cur = a;
  auto it = m.lower_bound(a);
  while (cur < b) {
    if (it == m.end() || it->first > cur) {
      const uint64_t e = (it == m.end()) ? b : std::min(b, it->first);
      it = m.emplace(cur, Seg{e, Acc{}, {}}).first;
    }
    out.push_back(it);
    cur = it->second.end;
    ++it;
  }
  return out;
}

bool ordered(const Acc& x, int s, const std::vector<uint64_t>& vc) {
  return x.stream < 0 || x.stream == s || comp(vc, x.stream) >= x.clk;
}

void report(const char* kind, uint64_t op, int s, uint64_t lo, uint64_t hi, const Acc& other, const char* okind) {
  State& st = S();
  if (st.races.size() >= 200) return;
  char buf[512];
  snprintf(buf, sizeof(buf), "%s of %s..%s by op %llu '%s' on %s is not ordered after the %s by op %llu '%s' on %s",
           kind, where(lo).c_str(), where(hi).c_str(), (unsigned long long)op, st.ops[op].name.c_str(),
           st.streams[s]->name.c_str(), okind, (unsigned long long)other.op, st.ops[other.op].name.c_str(),
           st.streams[other.stream]->name.c_str());
  st.races.push_back(buf);
}

void access(uint64_t op, int s, const std::vector<uint64_t>& vc, uint64_t a, uint64_t b, bool write) {
  if (b <= a) return;
  const uint64_t clk = comp(vc, s);
  for (auto it : cover(a, b)) {
    Seg& g = it->second;
    if (!ordered(g.w, s, vc)) report(write ? "write" : "read", op, s, it->first, g.end, g.w, "write");
    if (write) {
      for (const Acc& r : g.r)
        if (!ordered(r, s, vc)) report("write", op, s, it->first, g.end, r, "read");
      g.r.clear();
      g.w = Acc{s, clk, op};
    } else {
      bool found = false;
      for (Acc& r : g.r)
        if (r.stream == s) {
          r = Acc{s, clk, op};
          found = true;
        }
      if (!found) g.r.push_back(Acc{s, clk, op});
    }
  }
}

// Begin an operation on stream s: ordered after everything the host has
// waited for; advances the stream's own clock.
uint64_t begin_op(HbStream* hs, const std::string& name) {
  State& st = S();
  auto& v = st.vc[hs->id];
  join(v, st.vc[0]);
  if (v.size() <= (size_t)hs->id) v.resize(hs->id + 1, 0);
  v[hs->id] += 1;
  st.ops.push_back({name, hs->id});
  return st.ops.size() - 1;
}

}  // namespace

// --- checker API (hb.h) --------------------------------------------------------
void* hb_new_stream(const char* name) {
  State& st = S();
  HbStream* s = new HbStream{(int)st.streams.size(), name ? name : "stream"};
  st.streams.push_back(s);
  st.vc.push_back(std::vector<uint64_t>(s->id + 1, 0));
  return s;
}

void hb_op(hipStream_t stream, const char* name, const HbRanges& reads, const HbRanges& writes) {
  HbStream* hs = resolve(stream);
  const uint64_t op = begin_op(hs, name);
  const auto vc = S().vc[hs->id];
  for (auto& r : reads) access(op, hs->id, vc, r.first, r.second, false);
  for (auto& w : writes) access(op, hs->id, vc, w.first, w.second, true);
}

extern "C" {
void* tps_hb_new_stream(const char* name) { return hb_new_stream(name); }
void tps_hb_name_region(uint64_t start, uint64_t bytes, const char* name) {
  S().regions[start] = {start + bytes, name};
}
void tps_hb_host_access(uint64_t ptr, uint64_t bytes, int write) {
  State& st = S();
  st.vc[0][0] += 1;
  st.ops.push_back({write ? "host write" : "host read", 0});
  access(st.ops.size() - 1, 0, st.vc[0], ptr, ptr + bytes, write != 0);
}
void tps_hb_stream_access(void* stream, uint64_t ptr, uint64_t bytes, int write) {
  HbRanges none, r{{ptr, ptr + bytes}};
  hb_op(static_cast<hipStream_t>(stream), write ? "caller write" : "caller read", write ? none : r, write ? r : none);
}
void tps_hb_reset(void) {
  State& st = S();
  st.shadow.clear();
  st.races.clear();
}
int tps_hb_races(void) { return (int)S().races.size(); }
const char* tps_hb_report(void) {
  static std::string out;
  out.clear();
  for (auto& r : S().races) out += r + "\n";
  return out.c_str();
}
int64_t tps_hb_waits(void) { return S().waits; }
void tps_hb_drop_wait(int64_t n) { S().drop_wait = n; }
uint64_t tps_hb_ops(void) { return S().ops.size() - 1; }
int64_t tps_hb_count_ops(const char* name) {
  int64_t n = 0;
  for (auto& o : S().ops) n += o.name == name;
  return n;
}
}

// --- stand-in HIP runtime ------------------------------------------------------
hipError_t hipGetDevice(int* dev) {
  *dev = 0;
  return hipSuccess;
}
hipError_t hipSetDevice(int) { return hipSuccess; }
hipError_t hipDeviceGetAttribute(int* v, hipDeviceAttribute_t, int) {
  *v = 256;
  return hipSuccess;
}
hipError_t hipEventCreate(hipEvent_t* e) {
  *e = new HbEvent();
  return hipSuccess;
}
hipError_t hipEventCreateWithFlags(hipEvent_t* e, unsigned) { return hipEventCreate(e); }
hipError_t hipEventDestroy(hipEvent_t e) {
  delete e;
  return hipSuccess;
}
hipError_t hipEventRecord(hipEvent_t e, hipStream_t s) {
  HbStream* hs = resolve(s);
  begin_op(hs, "event record");
  e->vc = S().vc[hs->id];
  e->recorded = true;
  return hipSuccess;
}
hipError_t hipEventSynchronize(hipEvent_t e) {
  if (e->recorded) join(S().vc[0], e->vc);
  return hipSuccess;
}
hipError_t hipEventElapsedTime(float* ms, hipEvent_t, hipEvent_t) {
  *ms = 0.f;
  return hipSuccess;
}
hipError_t hipStreamWaitEvent(hipStream_t s, hipEvent_t e, unsigned) {
  State& st = S();
  const int64_t n = st.waits++;
  if (n == st.drop_wait) return hipSuccess;   // test hook: this wait is left out
  HbStream* hs = resolve(s);
  if (e->recorded) join(st.vc[hs->id], e->vc);
  return hipSuccess;
}
hipError_t hipStreamSynchronize(hipStream_t s) {
  join(S().vc[0], S().vc[resolve(s)->id]);
  return hipSuccess;
}
hipError_t hipStreamQuery(hipStream_t s) { return hipStreamSynchronize(s); }
hipError_t hipStreamDestroy(hipStream_t) { return hipSuccess; }
hipError_t hipStreamCreateWithFlags(hipStream_t* s, unsigned) {
  *s = static_cast<hipStream_t>(hb_new_stream("library stream"));
  return hipSuccess;
}
hipError_t hipExtStreamCreateWithCUMask(hipStream_t* s, uint32_t, const uint32_t*) {
  *s = static_cast<hipStream_t>(hb_new_stream("library queue stream"));
  return hipSuccess;
}
hipError_t hipMemcpyAsync(void* dst, const void* src, size_t bytes, hipMemcpyKind kind, hipStream_t s) {
  const char* name = kind == hipMemcpyDeviceToHost ? "copy device->host"
                     : kind == hipMemcpyHostToDevice ? "copy host->device" : "copy device->device";
  const uint64_t d = reinterpret_cast<uint64_t>(dst), r = reinterpret_cast<uint64_t>(src);
  hb_op(s, name, HbRanges{{r, r + bytes}}, HbRanges{{d, d + bytes}});
  return hipSuccess;
}
hipError_t hipMemcpy2DAsync(void* dst, size_t dpitch, const void* src, size_t spitch, size_t width, size_t height,
                            hipMemcpyKind kind, hipStream_t s) {
  const char* name = kind == hipMemcpyDeviceToHost ? "pitched copy device->host"
                     : kind == hipMemcpyHostToDevice ? "pitched copy host->device" : "pitched copy device->device";
  HbRanges rd, wr;
  const uint64_t d = reinterpret_cast<uint64_t>(dst), r = reinterpret_cast<uint64_t>(src);
  for (size_t i = 0; i < height; ++i) {
    rd.push_back({r + i * spitch, r + i * spitch + width});
    wr.push_back({d + i * dpitch, d + i * dpitch + width});
  }
  hb_op(s, name, rd, wr);
  return hipSuccess;
}
hipError_t hipHostMalloc(void** p, size_t bytes, unsigned) {
  *p = malloc(bytes ? bytes : 1);
  return *p ? hipSuccess : hipErrorInvalidValue;
}
hipError_t hipHostFree(void* p) {
  free(p);
  return hipSuccess;
}
hipError_t hipGetLastError(void) { return hipSuccess; }
const char* hipGetErrorString(hipError_t) { return "stand-in runtime error"; }
