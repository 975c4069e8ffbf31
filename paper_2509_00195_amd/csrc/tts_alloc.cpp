// Roofline-guided split of the KV-cache memory between the verifier
// (prefill) and the generator (decode) (Sec. 4.3): choose the batch sizes
// that minimise the modelled total time of N requests under one memory
// budget, by a linear search over the prefill batch size with the decode
// batch size on the memory boundary.
#include <cmath>
#include <cstdint>

#include "tts.h"

namespace tts {

// Roofline time of one batch: max(FLOPs / P, bytes / BW).
static double roof(double flops, double bytes, double peak_flops, double peak_bw) {
  return std::fmax(flops / peak_flops, bytes / peak_bw);
}

// Prefill of b sequences of s tokens: dense layers 2 * params flops per
// token, causal attention 2 * d * s * (s + 1) flops per layer and sequence
// (s (s + 1) / 2 query-key pairs, a d-long product for the scores and one
// for the values); bytes: the weights once plus the KV written.
static double t_prefill(const tts_model_cost& m, double b, double s, double pf, double bw) {
  const double flops = 2.0 * m.params * b * s + 2.0 * m.num_layers * m.attn_dim * b * s * (s + 1.0);
  const double bytes = m.weight_bytes + b * m.kv_bytes_per_token * s;
  return roof(flops, bytes, pf, bw);
}

// One decode step of b sequences over caches of c tokens: 2 * params flops
// per token, 4 * d * c attention flops per layer and sequence; bytes: the
// weights once plus the KV read.
static double t_decode(const tts_model_cost& m, double b, double c, double pf, double bw) {
  const double flops = 2.0 * m.params * b + 4.0 * m.num_layers * m.attn_dim * b * c;
  const double bytes = m.weight_bytes + b * m.kv_bytes_per_token * c;
  return roof(flops, bytes, pf, bw);
}

// Modelled time of one (b_pre, b_dec) choice (both >= 1).
void alloc_time(const tts_alloc_problem& pr, int64_t b_pre, int64_t b_dec, tts_alloc_result* out) {
  const double n = static_cast<double>(pr.num_requests);
  const double s = static_cast<double>(pr.verify_len), sd = static_cast<double>(pr.decode_len);
  const double tp = t_prefill(pr.verifier, static_cast<double>(b_pre), s, pr.peak_flops, pr.peak_bw);
  const double td = t_decode(pr.generator, static_cast<double>(b_dec), sd / 2.0, pr.peak_flops, pr.peak_bw);
  out->b_pre = b_pre;
  out->b_dec = b_dec;
  out->t_pre = std::ceil(n / static_cast<double>(b_pre)) * tp;
  out->t_dec = std::ceil(n / static_cast<double>(b_dec)) * sd * td;
  out->t_tot = out->t_pre + out->t_dec;
}

// The search; false when no feasible pair exists.
bool alloc_search(const tts_alloc_problem& pr, tts_alloc_result* out) {
  const double kv_pre = pr.verifier.kv_bytes_per_token * static_cast<double>(pr.verify_len);
  const double kv_dec = pr.generator.kv_bytes_per_token * static_cast<double>(pr.decode_len);
  // Every feasible prefill batch (at most N, leaving room for one decode
  // sequence); the decode batch fills the rest of the budget (at most N).
  const double room = std::floor((pr.mem_bytes - kv_dec) / kv_pre);
  if (!(room >= 1.0)) return false;
  const int64_t max_pre = static_cast<int64_t>(std::fmin(room, static_cast<double>(pr.num_requests)));
  bool have = false;
  tts_alloc_result best{};
  for (int64_t bp = 1; bp <= max_pre; ++bp) {
    const double fit = std::floor((pr.mem_bytes - static_cast<double>(bp) * kv_pre) / kv_dec);
    const int64_t bd = static_cast<int64_t>(std::fmin(fit, static_cast<double>(pr.num_requests)));
    if (bd < 1) continue;
    tts_alloc_result r;
    alloc_time(pr, bp, bd, &r);
    // Ties go to the larger decode batch (decoding is the more
    // memory-sensitive stage).
    if (!have || r.t_tot < best.t_tot || (r.t_tot == best.t_tot && bd > best.b_dec)) {
      best = r;
      have = true;
    }
  }
  if (have) *out = best;
  return have;
}

}  // namespace tts
