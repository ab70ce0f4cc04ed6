// Optional per-kernel event timing for diagnostics (mebp_kernel_timing*): when enabled,
// every instrumented launch is bracketed by a pair of HIP events from a pool created at
// enable time, tagged with the kernel's name and its algorithmic flops and bytes. The
// report synchronises on the recorded events and aggregates per kernel name.
// mebp_kernel_repeat makes every launch of one named kernel run several times back to
// back; with timing enabled the whole burst is bracketed by one event pair and counted as
// that many launches, so the report gives the kernel's back-to-back in-stream duration
// without the event and dispatch latency that a pair around a single launch includes.
// Not thread-safe: configure, run and report from one host thread.
#include <stdio.h>
#include <string.h>

#include <map>
#include <string>
#include <vector>

#include "mebp_internal.h"

namespace mebp {
namespace {
struct Rec {
  const char* name;
  double flops, bytes;
  int idx, count;
};
struct State {
  bool on = false;
  std::vector<hipEvent_t> ev;  // 2 per record
  std::vector<Rec> recs;
  std::string repeat_name;  // launches of this kernel run repeat_times times in a row
  int repeat_times = 1;
};
State& S() {
  static State s;
  return s;
}
}  // namespace

int timer_begin(hipStream_t st, const char* name, double flops, double bytes, int count) {
  State& s = S();
  if (!s.on || 2 * (s.recs.size() + 1) > s.ev.size()) return -1;
  const int idx = (int)s.recs.size();
  s.recs.push_back({name, flops * count, bytes * count, idx, count});
  (void)hipEventRecord(s.ev[2 * idx], st);
  return idx;
}
void timer_end(hipStream_t st, int idx) {
  if (idx >= 0) (void)hipEventRecord(S().ev[2 * idx + 1], st);
}

int repeat_count(const char* name) {
  const State& s = S();
  return (s.repeat_times > 1 && s.repeat_name == name) ? s.repeat_times : 1;
}

int set_repeat(const char* name, int times) {
  State& s = S();
  if (!name || times <= 1) {
    s.repeat_name.clear();
    s.repeat_times = 1;
    return 0;
  }
  // kernels that update a buffer they also read (in place) would not give the same result
  // twice in a row
  static const char* const in_place[] = {
      "gemm_tn_act_bwd", "splitk_finalize_actbwd",  // fp16 g, u -> bf16 dg, du
      "rope_fwd", "qkv_post", "headnorm_bwd",       // q, k (or dq, dk) rotated / normalised
      "ce_chunk_stats", "ce_probs", "ce_dh_accum", "ce_final",  // LM-head running state
      "lora_adamw", "lora_grad_accumulate"};        // parameters, moments, accumulators
  for (const char* n : in_place)
    if (!strcmp(name, n)) return -1;
  s.repeat_name = name;
  s.repeat_times = times;
  return 0;
}

int timing_enable(int enable, int capacity) {
  State& s = S();
  for (hipEvent_t e : s.ev) (void)hipEventDestroy(e);
  s.ev.clear();
  s.recs.clear();
  s.on = false;
  if (!enable) return 0;
  s.ev.resize(2 * (size_t)capacity);
  for (auto& e : s.ev)
    if (hipEventCreate(&e) != hipSuccess) return -1;
  s.on = true;
  return 0;
}

int timing_report(char* buf, size_t len) {
  State& s = S();
  struct Agg {
    int n = 0;
    double ms = 0, flops = 0, bytes = 0;
  };
  std::map<std::string, Agg> agg;
  for (const Rec& r : s.recs) {
    float ms = 0.f;
    if (hipEventSynchronize(s.ev[2 * r.idx + 1]) != hipSuccess) return -1;
    if (hipEventElapsedTime(&ms, s.ev[2 * r.idx], s.ev[2 * r.idx + 1]) != hipSuccess) return -1;
    Agg& a = agg[r.name];
    a.n += r.count;
    a.ms += ms;
    a.flops += r.flops;
    a.bytes += r.bytes;
  }
  std::string out = "[";
  char line[512];
  bool first = true;
  for (auto& kv : agg) {
    snprintf(line, sizeof line, "%s{\"kernel\":\"%s\",\"launches\":%d,\"ms\":%.6f,\"flops\":%.6e,\"bytes\":%.6e}",
             first ? "" : ",", kv.first.c_str(), kv.second.n, kv.second.ms, kv.second.flops, kv.second.bytes);
    out += line;
    first = false;
  }
  out += "]";
  if (buf && len) {
    strncpy(buf, out.c_str(), len - 1);
    buf[len - 1] = 0;
  }
  return (int)out.size() + 1;
}

}  // namespace mebp
