// Event-pair kernel timing behind bi_profile_begin / bi_profile_end.
#include <cstring>
#include <map>
#include <string>
#include <vector>

#include "internal.h"
#include "profile.h"

namespace bi {
namespace {

struct Pair {
    const char *name;
    hipEvent_t a, b;
};

bool g_on = false;
std::vector<Pair> g_pairs;
std::vector<hipEvent_t> g_pool;
size_t g_used = 0;

hipEvent_t take()
{
    if (g_used == g_pool.size()) {
        hipEvent_t e;
        if (hipEventCreate(&e) != hipSuccess) return nullptr;
        g_pool.push_back(e);
    }
    return g_pool[g_used++];
}

}  // namespace

bool profiling() { return g_on; }

void prof_mark(const char *name, hipStream_t s, bool end)
{
    if (!g_on) return;
    if (!end) {
        hipEvent_t e = take();
        if (!e) return;
        hipEventRecord(e, s);
        g_pairs.push_back({name, e, nullptr});
    } else if (!g_pairs.empty() && g_pairs.back().b == nullptr) {
        hipEvent_t e = take();
        if (!e) return;
        hipEventRecord(e, s);
        g_pairs.back().b = e;
    }
}

}  // namespace bi

extern "C" {

int bi_profile_begin(void)
{
    bi::g_pairs.clear();
    bi::g_used = 0;
    bi::g_on = true;
    return BI_OK;
}

int bi_profile_end(bi_profile_entry *out, int32_t cap, int32_t *n_out)
{
    bi::g_on = false;
    if (!n_out || (cap > 0 && !out)) return bi::fail(BI_ERR_INVALID_ARG, "out / n_out is NULL");
    std::map<std::string, std::pair<int64_t, double>> acc;
    for (const auto &p : bi::g_pairs) {
        if (!p.b) continue;
        if (hipEventSynchronize(p.b) != hipSuccess) return bi::fail(BI_ERR_DEVICE, "hipEventSynchronize failed");
        float ms = 0.0f;
        if (hipEventElapsedTime(&ms, p.a, p.b) != hipSuccess)
            return bi::fail(BI_ERR_DEVICE, "hipEventElapsedTime failed");
        auto &e = acc[p.name];
        e.first += 1;
        e.second += ms;
    }
    int32_t n = 0;
    for (const auto &kv : acc) {
        if (n < cap) {
            std::memset(out[n].name, 0, sizeof(out[n].name));
            std::strncpy(out[n].name, kv.first.c_str(), sizeof(out[n].name) - 1);
            out[n].launches = kv.second.first;
            out[n].total_ms = kv.second.second;
        }
        ++n;
    }
    *n_out = n;
    bi::g_pairs.clear();
    bi::g_used = 0;
    return BI_OK;
}

}  // extern "C"
