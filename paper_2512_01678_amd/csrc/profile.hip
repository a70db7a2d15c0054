// profile.hip -- HIP-event timing of individual launches (benchmark support).
//
// When enabled, every aggregation / GEMM launcher records an event pair on its
// stream around the kernel(s) it enqueues.  Events come from a fixed pool
// created at enable time; records beyond the capacity overwrite the oldest.
#include <cstring>
#include <mutex>
#include <vector>

#include "internal.h"

namespace gcn {
namespace {

struct Record {
  gcn_profile_record meta;
  hipEvent_t start = nullptr, stop = nullptr;
};

std::mutex g_mu;
std::vector<Record> g_ring;
int64_t g_next = 0;  // total records started
bool g_on = false;
char g_only[64] = "";  // record only this family when non-empty

}  // namespace

ProfScope::ProfScope(const char* name, int32_t width, int64_t rows, int64_t nnz, hipStream_t s) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_on || g_ring.empty()) return;
  if (g_only[0] && strcmp(g_only, name) != 0) return;
  slot = (int)(g_next % (int64_t)g_ring.size());
  ++g_next;
  Record& r = g_ring[slot];
  snprintf(r.meta.name, sizeof r.meta.name, "%s", name);
  r.meta.width = width;
  r.meta.rows = rows;
  r.meta.nnz = nnz;
  r.meta.ms = -1.f;
  stream = s;
  (void)hipEventRecord(r.start, s);
}

ProfScope::~ProfScope() {
  if (slot < 0) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (slot < (int)g_ring.size()) (void)hipEventRecord(g_ring[slot].stop, stream);
}

}  // namespace gcn

using namespace gcn;

extern "C" gcn_status gcn_profile_enable(int32_t capacity) {
  std::lock_guard<std::mutex> lk(g_mu);
  for (Record& r : g_ring) {
    (void)hipEventDestroy(r.start);
    (void)hipEventDestroy(r.stop);
  }
  g_ring.clear();
  g_next = 0;
  g_on = false;
  if (capacity < 0) return fail(GCN_E_INVALID, "gcn_profile_enable: negative capacity");
  if (capacity == 0) return GCN_OK;
  g_ring.resize((size_t)capacity);
  for (Record& r : g_ring) {
    GCN_HIP(hipEventCreate(&r.start), "profile event");
    GCN_HIP(hipEventCreate(&r.stop), "profile event");
  }
  g_on = true;
  return GCN_OK;
}

extern "C" int32_t gcn_profile_count(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  return (int32_t)std::min<int64_t>(g_next, (int64_t)g_ring.size());
}

extern "C" gcn_status gcn_profile_read(int32_t i, gcn_profile_record* rec) {
  std::lock_guard<std::mutex> lk(g_mu);
  const int64_t held = std::min<int64_t>(g_next, (int64_t)g_ring.size());
  if (!rec || i < 0 || i >= held) return fail(GCN_E_INVALID, "gcn_profile_read: index out of range");
  const int64_t first = g_next - held;
  Record& r = g_ring[(size_t)((first + i) % (int64_t)g_ring.size())];
  GCN_HIP(hipEventSynchronize(r.stop), "profile sync");
  float ms = 0.f;
  GCN_HIP(hipEventElapsedTime(&ms, r.start, r.stop), "profile elapsed");
  r.meta.ms = ms;
  *rec = r.meta;
  return GCN_OK;
}

extern "C" gcn_status gcn_profile_only(const char* name) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (name && strlen(name) >= sizeof g_only) return fail(GCN_E_INVALID, "gcn_profile_only: name too long");
  snprintf(g_only, sizeof g_only, "%s", name ? name : "");
  return GCN_OK;
}

extern "C" gcn_status gcn_profile_reset(void) {
  std::lock_guard<std::mutex> lk(g_mu);
  g_next = 0;
  return GCN_OK;
}
