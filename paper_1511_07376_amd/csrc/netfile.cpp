// NetFile parser.  The paper's engine is configured by a plain-text file that
// lists the layers of the trained model in order, with their settings, and
// three engine parameters: allocated_ram, execution_mode and auto_tuning
// (Sec. 3.2).  Its exact syntax is in a figure that is not reproduced, so the
// syntax here is this library's own; it is documented with cnn_netfile_parse
// in cnn.h.  The parser fills cnn_layer_desc records (weights left NULL: the
// caller binds its device parameters) and a cnn_netfile_config.
#include <cerrno>
#include <cmath>
#include <cstdlib>
#include <cstring>
#include <string>
#include <vector>

#include "common.h"

namespace cnn {
namespace {

struct Parser {
    int line = 0;

    int err(int status, const char* fmt, const std::string& a = "", const std::string& b = "") {
        char msg[256];
        snprintf(msg, sizeof(msg), fmt, a.c_str(), b.c_str());
        return fail(status, "netfile line %d: %s", line, msg);
    }

    // Whole-token integer in [lo, hi].
    bool to_int(const std::string& s, long lo, long hi, int* out) {
        if (s.empty()) return false;
        errno = 0;
        char* end = nullptr;
        const long v = strtol(s.c_str(), &end, 10);
        if (errno || *end != '\0' || v < lo || v > hi) return false;
        *out = (int)v;
        return true;
    }

    // "7" or "7x5" (height x width).
    bool to_pair(const std::string& s, long lo, int* h, int* w) {
        const size_t x = s.find('x');
        if (x == std::string::npos) {
            if (!to_int(s, lo, 1 << 20, h)) return false;
            *w = *h;
            return true;
        }
        return to_int(s.substr(0, x), lo, 1 << 20, h) && to_int(s.substr(x + 1), lo, 1 << 20, w);
    }

    bool to_float(const std::string& s, float* out) {
        if (s.empty()) return false;
        errno = 0;
        char* end = nullptr;
        const float v = strtof(s.c_str(), &end);
        if (errno || *end != '\0' || !std::isfinite(v)) return false;
        *out = v;
        return true;
    }
};

std::vector<std::string> split_words(const std::string& line) {
    std::vector<std::string> words;
    size_t i = 0;
    while (i < line.size()) {
        while (i < line.size() && isspace((unsigned char)line[i])) ++i;
        size_t j = i;
        while (j < line.size() && !isspace((unsigned char)line[j])) ++j;
        if (j > i) words.push_back(line.substr(i, j - i));
        i = j;
    }
    return words;
}

// Parses the options of one layer statement ("key=value" or a bare flag) into
// d.  allowed: the keys and flags this layer type takes.
int parse_layer(Parser& ps, const std::vector<std::string>& words, size_t first,
                const std::vector<std::string>& allowed, cnn_layer_desc& d, bool* seen_out,
                bool* seen_kernel) {
    std::vector<std::string> seen;
    for (size_t i = first; i < words.size(); ++i) {
        const std::string& wd = words[i];
        const size_t eq = wd.find('=');
        const std::string key = eq == std::string::npos ? wd : wd.substr(0, eq);
        const std::string val = eq == std::string::npos ? "" : wd.substr(eq + 1);
        bool ok_key = false;
        for (const auto& a : allowed) ok_key |= (a == key);
        if (!ok_key) return ps.err(CNN_ERR_INVALID, "unknown option '%s' for '%s'", key, words[0]);
        for (const auto& s : seen)
            if (s == key) return ps.err(CNN_ERR_INVALID, "option '%s' given twice", key);
        seen.push_back(key);
        const bool flag = (key == "relu");
        if (flag != (eq == std::string::npos))
            return ps.err(CNN_ERR_INVALID, flag ? "'%s' takes no value" : "option '%s' needs a value", key);
        bool ok = true;
        if (key == "relu") {
            d.fuse_relu = 1;
        } else if (key == "out") {
            ok = ps.to_int(val, 1, 0x7fffffff, &d.out_channels);
            *seen_out = true;
        } else if (key == "in") {
            ok = ps.to_int(val, 1, 0x7fffffff, d.type == CNN_LAYER_FC ? &d.in_features : &d.in_channels);
        } else if (key == "kernel") {
            ok = ps.to_pair(val, 1, &d.kernel_h, &d.kernel_w);
            *seen_kernel = true;
        } else if (key == "stride") {
            ok = ps.to_pair(val, 1, &d.stride_h, &d.stride_w);
        } else if (key == "pad") {
            ok = ps.to_pair(val, 0, &d.pad_h, &d.pad_w);
        } else if (key == "groups") {
            ok = ps.to_int(val, 1, 1 << 20, &d.groups);
        } else if (key == "ceil") {
            ok = ps.to_int(val, 0, 1, &d.ceil_mode);
        } else if (key == "size") {
            ok = ps.to_int(val, 1, 1 << 20, &d.lrn_size);
        } else if (key == "alpha") {
            ok = ps.to_float(val, &d.lrn_alpha);
        } else if (key == "beta") {
            ok = ps.to_float(val, &d.lrn_beta);
        } else if (key == "k") {
            ok = ps.to_float(val, &d.lrn_k);
        }
        if (!ok) return ps.err(CNN_ERR_INVALID, "bad value '%s' for option '%s'", val, key);
    }
    return CNN_OK;
}

int parse(const char* text, cnn_layer_desc* layers, int max_layers, int* n_layers,
          cnn_netfile_config* cfg) {
    Parser ps;
    cnn_netfile_config c{};
    c.execution_mode = CNN_EXEC_PARALLEL;
    int count = 0;
    const char* p = text;
    while (*p) {
        const char* e = strchr(p, '\n');
        std::string line = e ? std::string(p, (size_t)(e - p)) : std::string(p);
        p = e ? e + 1 : p + line.size();
        ++ps.line;
        const size_t hash = line.find('#');
        if (hash != std::string::npos) line.resize(hash);
        std::vector<std::string> w = split_words(line);
        if (w.empty()) continue;
        std::string head = w[0];
        if (head.size() > 1 && head.back() == ':') head.pop_back();  // "key: value" form

        // ---- engine parameters
        if (head == "input") {
            if (w.size() != 4 || !ps.to_int(w[1], 1, 1 << 24, &c.in_channels) ||
                !ps.to_int(w[2], 1, 1 << 24, &c.in_height) || !ps.to_int(w[3], 1, 1 << 24, &c.in_width))
                return ps.err(CNN_ERR_INVALID, "'input' needs three positive integers C H W");
            continue;
        }
        if (head == "execution_mode" || head == "auto_tuning" || head == "allocated_ram") {
            if (w.size() != 2) return ps.err(CNN_ERR_INVALID, "'%s' needs one value", head);
            const std::string& v = w[1];
            if (head == "execution_mode") {
                if (v == "parallel") c.execution_mode = CNN_EXEC_PARALLEL;
                else if (v == "graph") c.execution_mode = CNN_EXEC_GRAPH;
                else if (v == "sequential")
                    return ps.err(CNN_ERR_UNSUPPORTED,
                                  "execution_mode '%s': this library runs every layer on the GPU", v);
                else return ps.err(CNN_ERR_INVALID, "execution_mode '%s' (parallel or graph)", v);
            } else if (head == "auto_tuning") {
                if (v == "on" || v == "true" || v == "1") c.auto_tuning = 1;
                else if (v == "off" || v == "false" || v == "0") c.auto_tuning = 0;
                else return ps.err(CNN_ERR_INVALID, "auto_tuning '%s' (on or off)", v);
            } else {
                int mib;
                if (!ps.to_int(v, 0, 0x7fffffff, &mib))
                    return ps.err(CNN_ERR_INVALID, "allocated_ram '%s' (MiB, >= 0)", v);
                c.allocated_ram_mib = mib;
            }
            continue;
        }

        // ---- layers
        cnn_layer_desc d{};
        d.groups = 1;
        d.stride_h = d.stride_w = 1;
        d.ceil_mode = 1;
        d.lrn_size = 5;
        d.lrn_alpha = 1e-4f;
        d.lrn_beta = 0.75f;
        d.lrn_k = 1.0f;
        bool seen_out = false, seen_kernel = false;
        int rc = CNN_OK;
        if (head == "conv") {
            d.type = CNN_LAYER_CONV;
            rc = parse_layer(ps, w, 1, {"out", "in", "kernel", "stride", "pad", "groups", "relu"}, d,
                             &seen_out, &seen_kernel);
            if (!rc && (!seen_out || !seen_kernel))
                return ps.err(CNN_ERR_INVALID, "conv needs out= and kernel=");
        } else if (head == "fc") {
            d.type = CNN_LAYER_FC;
            rc = parse_layer(ps, w, 1, {"out", "in", "relu"}, d, &seen_out, &seen_kernel);
            if (!rc && !seen_out) return ps.err(CNN_ERR_INVALID, "fc needs out=");
        } else if (head == "pool") {
            d.type = CNN_LAYER_POOL;
            if (w.size() < 2 || (w[1] != "max" && w[1] != "avg"))
                return ps.err(CNN_ERR_INVALID, "pool needs a mode, max or avg, first");
            d.pool_mode = w[1] == "max" ? CNN_POOL_MAX : CNN_POOL_AVG;
            rc = parse_layer(ps, w, 2, {"kernel", "stride", "pad", "ceil", "relu"}, d, &seen_out,
                             &seen_kernel);
            if (!rc && !seen_kernel) return ps.err(CNN_ERR_INVALID, "pool needs kernel=");
        } else if (head == "lrn") {
            d.type = CNN_LAYER_LRN;
            rc = parse_layer(ps, w, 1, {"size", "alpha", "beta", "k"}, d, &seen_out, &seen_kernel);
        } else if (head == "relu" || head == "softmax") {
            d.type = head == "relu" ? CNN_LAYER_RELU : CNN_LAYER_SOFTMAX;
            if (w.size() != 1) return ps.err(CNN_ERR_INVALID, "'%s' takes no options", head);
        } else {
            return ps.err(CNN_ERR_INVALID, "unknown statement '%s'", head);
        }
        if (rc) return rc;
        if (layers) {
            if (count >= max_layers)
                return ps.err(CNN_ERR_INVALID, "more layers than the %s entries provided",
                              std::to_string(max_layers));
            layers[count] = d;
        }
        ++count;
    }
    *n_layers = count;
    *cfg = c;
    return CNN_OK;
}

}  // namespace
}  // namespace cnn

extern "C" int cnn_netfile_parse(const char* text, cnn_layer_desc* layers, int max_layers,
                                 int* n_layers, cnn_netfile_config* config) {
    if (!text || !n_layers || !config) return cnn::fail(CNN_ERR_INVALID, "netfile: null argument");
    if (layers && max_layers < 0) return cnn::fail(CNN_ERR_INVALID, "netfile: max_layers %d", max_layers);
    return cnn::parse(text, layers, max_layers, n_layers, config);
}
