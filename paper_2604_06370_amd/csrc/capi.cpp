// C-ABI glue: error reporting, argument validation shared by the attention entry
// points, and the host-side RoPE table.
#include <cmath>
#include <string>

#include "internal.hpp"

namespace {
thread_local std::string g_last_error;
}

namespace fkv {

fkv_status fail(fkv_status code, const std::string &msg) {
    g_last_error = msg;
    return code;
}

void clear_error() { g_last_error.clear(); }

int64_t plan_max_pages(const fkv_plan *plan) { return plan ? plan->max_pages_used : 0; }

// Checks shared by decode and prefill: pointers present, supported shapes.
fkv_status validate_attn_common(const fkv_attn_args *a, const char *who) {
    const std::string w(who);
    if (!a) return fail(FKV_ERR_INVALID, w + ": null args");
    if (!a->q || !a->base_kv || !a->base_bt || !a->seq_lens || !a->out)
        return fail(FKV_ERR_INVALID, w + ": q, base_kv, base_bt, seq_lens and out are required");
    if (a->n_agents < 1 || a->hq < 1 || a->hkv < 1 || a->max_pages < 1)
        return fail(FKV_ERR_INVALID, w + ": n_agents, hq, hkv and max_pages must be positive");
    if (a->hq % a->hkv) return fail(FKV_ERR_INVALID, w + ": hq must be a multiple of hkv");
    if (a->d != 128) return fail(FKV_ERR_UNSUPPORTED, w + ": only head dim 128 is implemented");
    if (a->page_size != 16) return fail(FKV_ERR_UNSUPPORTED, w + ": only page size 16 is implemented");
    if (a->r != 0 && a->r != 8 && a->r != 16 && a->r != 32 && a->r != 64)
        return fail(FKV_ERR_UNSUPPORTED, w + ": rank must be 0, 8, 16, 32 or 64");
    if (a->r > 0 && (!a->res_kv || !a->res_bt || !a->lora_b || !a->adapter_idx))
        return fail(FKV_ERR_INVALID, w + ": res_kv, res_bt, lora_b and adapter_idx are required when r > 0");
    if ((a->rope_cos == nullptr) != (a->rope_sin == nullptr))
        return fail(FKV_ERR_INVALID, w + ": rope_cos and rope_sin must both be given or both be NULL");
    if (a->rope_cos && a->rope_max_pos < 1) return fail(FKV_ERR_INVALID, w + ": rope_max_pos must be positive");
    if (!(a->scale > 0.f) || !std::isfinite(a->scale)) return fail(FKV_ERR_INVALID, w + ": scale must be a positive finite number");
    return FKV_OK;
}

}  // namespace fkv

extern "C" {

const char *fkv_last_error(void) { return g_last_error.c_str(); }

const char *fkv_version(void) { return "forkkv-mi355x 0.2 (gfx950)"; }

fkv_status fkv_validate_tables(const int32_t *base_bt, const int32_t *res_bt, const int32_t *seq_lens,
                               const int32_t *adapter_idx, int32_t n_agents, int32_t max_pages, int32_t page_size,
                               int32_t num_base_pages, int32_t num_res_pages) {
    fkv::clear_error();
    if (!base_bt || !seq_lens || n_agents < 1 || max_pages < 1 || page_size < 1 || num_base_pages < 1)
        return fkv::fail(FKV_ERR_INVALID, "fkv_validate_tables: bad argument");
    for (int32_t a = 0; a < n_agents; ++a) {
        const int64_t L = seq_lens[a];
        if (L < 1 || L > (int64_t)max_pages * page_size)
            return fkv::fail(FKV_ERR_INVALID, "fkv_validate_tables: agent " + std::to_string(a) + " has length " +
                                                  std::to_string(L));
        const int32_t np = (int32_t)((L + page_size - 1) / page_size);
        const bool res = res_bt && adapter_idx && adapter_idx[a] >= 0;
        for (int32_t i = 0; i < np; ++i) {
            const int32_t b = base_bt[(int64_t)a * max_pages + i];
            if (b < 0 || b >= num_base_pages)
                return fkv::fail(FKV_ERR_INVALID, "fkv_validate_tables: agent " + std::to_string(a) + " page " +
                                                      std::to_string(i) + " names base page " + std::to_string(b));
            if (res) {
                const int32_t r = res_bt[(int64_t)a * max_pages + i];
                if (r < 0 || r >= num_res_pages)
                    return fkv::fail(FKV_ERR_INVALID, "fkv_validate_tables: agent " + std::to_string(a) + " page " +
                                                          std::to_string(i) + " names residual page " + std::to_string(r));
            }
        }
    }
    return FKV_OK;
}

fkv_status fkv_rope_table(int32_t d, int32_t max_pos, double base, float *cos_out, float *sin_out) {
    fkv::clear_error();
    if (d != 128 || max_pos < 16 || max_pos % 16 || !(base > 0.0) || !cos_out || !sin_out)
        return fkv::fail(FKV_ERR_INVALID, "fkv_rope_table: needs d = 128 and max_pos a positive multiple of 16");
    const int32_t half = d / 2;
    for (int32_t i = 0; i < half; ++i) {
        const double inv_freq = std::pow(base, -2.0 * (double)i / (double)d);
        // pair i = 16*mt + 4*grp + k of position 16*page + t sits at [page][mt][t + 16*grp][k]
        const int32_t mt = i / 16, grp = (i % 16) / 4, k = i % 4;
        for (int32_t p = 0; p < max_pos; ++p) {
            const double ang = (double)p * inv_freq;
            const int64_t off = (int64_t)(p / 16) * 1024 + mt * 256 + (p % 16 + 16 * grp) * 4 + k;
            cos_out[off] = (float)std::cos(ang);
            sin_out[off] = (float)std::sin(ang);
        }
    }
    return FKV_OK;
}

}  // extern "C"
