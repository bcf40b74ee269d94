// A small, bounds-checked JSON reader: enough for the header of a
// safetensors file (objects, arrays, strings, integers, true/false/null).
// Host-only.
#pragma once

#include <cstdint>
#include <map>
#include <memory>
#include <string>
#include <vector>

namespace sllm {
namespace json {

struct Value {
    enum Kind { Null, Bool, Number, String, Array, Object } kind = Null;
    bool b = false;
    bool integral = false;   // the number had no fraction or exponent
    bool negative = false;
    uint64_t u = 0;          // magnitude of an integral number (if it fits)
    bool fits = true;        // integral magnitude fits in 64 bits
    std::string s;
    std::vector<Value> items;                          // Array
    std::vector<std::pair<std::string, Value>> fields; // Object, in source order

    const Value* get(const std::string& key) const {
        for (const auto& f : fields)
            if (f.first == key) return &f.second;
        return nullptr;
    }
};

class Parser {
  public:
    Parser(const char* p, size_t n) : p_(p), n_(n) {}

    // Parse one document; false (with error()) on malformed input or
    // nesting deeper than 32.
    bool parse(Value* out) {
        skip_ws();
        if (!value(out, 0)) return false;
        skip_ws();
        if (i_ != n_) return err("trailing bytes after the JSON value");
        return true;
    }
    const std::string& error() const { return err_; }

  private:
    const char* p_;
    size_t n_, i_ = 0;
    std::string err_;

    bool err(const char* m) {
        if (err_.empty()) err_ = std::string(m) + " at byte " + std::to_string(i_);
        return false;
    }
    void skip_ws() {
        while (i_ < n_ && (p_[i_] == ' ' || p_[i_] == '\t' || p_[i_] == '\n' || p_[i_] == '\r')) ++i_;
    }
    bool lit(const char* w) {
        size_t k = 0;
        while (w[k]) {
            if (i_ + k >= n_ || p_[i_ + k] != w[k]) return err("bad literal");
            ++k;
        }
        i_ += k;
        return true;
    }
    static void put_utf8(std::string& s, uint32_t c) {
        if (c < 0x80) {
            s.push_back((char)c);
        } else if (c < 0x800) {
            s.push_back((char)(0xC0 | (c >> 6)));
            s.push_back((char)(0x80 | (c & 0x3F)));
        } else if (c < 0x10000) {
            s.push_back((char)(0xE0 | (c >> 12)));
            s.push_back((char)(0x80 | ((c >> 6) & 0x3F)));
            s.push_back((char)(0x80 | (c & 0x3F)));
        } else {
            s.push_back((char)(0xF0 | (c >> 18)));
            s.push_back((char)(0x80 | ((c >> 12) & 0x3F)));
            s.push_back((char)(0x80 | ((c >> 6) & 0x3F)));
            s.push_back((char)(0x80 | (c & 0x3F)));
        }
    }
    bool hex4(uint32_t* out) {
        if (n_ - i_ < 4) return err("short \\u escape");
        uint32_t v = 0;
        for (int k = 0; k < 4; ++k) {
            const char c = p_[i_++];
            v <<= 4;
            if (c >= '0' && c <= '9') v |= (uint32_t)(c - '0');
            else if (c >= 'a' && c <= 'f') v |= (uint32_t)(c - 'a' + 10);
            else if (c >= 'A' && c <= 'F') v |= (uint32_t)(c - 'A' + 10);
            else return err("bad \\u escape");
        }
        *out = v;
        return true;
    }
    bool string(std::string* out) {
        if (i_ >= n_ || p_[i_] != '"') return err("expected a string");
        ++i_;
        out->clear();
        while (true) {
            if (i_ >= n_) return err("unterminated string");
            const char c = p_[i_++];
            if (c == '"') return true;
            if ((unsigned char)c < 0x20) return err("control character in string");
            if (c != '\\') {
                out->push_back(c);
                continue;
            }
            if (i_ >= n_) return err("unterminated escape");
            const char e = p_[i_++];
            switch (e) {
                case '"': out->push_back('"'); break;
                case '\\': out->push_back('\\'); break;
                case '/': out->push_back('/'); break;
                case 'b': out->push_back('\b'); break;
                case 'f': out->push_back('\f'); break;
                case 'n': out->push_back('\n'); break;
                case 'r': out->push_back('\r'); break;
                case 't': out->push_back('\t'); break;
                case 'u': {
                    uint32_t c1 = 0;
                    if (!hex4(&c1)) return false;
                    if (c1 >= 0xD800 && c1 < 0xDC00) {  // surrogate pair
                        uint32_t c2 = 0;
                        if (n_ - i_ < 2 || p_[i_] != '\\' || p_[i_ + 1] != 'u') return err("lone surrogate");
                        i_ += 2;
                        if (!hex4(&c2) || c2 < 0xDC00 || c2 >= 0xE000) return err("bad surrogate pair");
                        c1 = 0x10000 + ((c1 - 0xD800) << 10) + (c2 - 0xDC00);
                    } else if (c1 >= 0xDC00 && c1 < 0xE000) {
                        return err("lone surrogate");
                    }
                    put_utf8(*out, c1);
                    break;
                }
                default: return err("bad escape");
            }
        }
    }
    bool number(Value* v) {
        v->kind = Value::Number;
        v->integral = true;
        if (i_ < n_ && p_[i_] == '-') {
            v->negative = true;
            ++i_;
        }
        if (i_ >= n_ || p_[i_] < '0' || p_[i_] > '9') return err("bad number");
        if (p_[i_] == '0' && i_ + 1 < n_ && p_[i_ + 1] >= '0' && p_[i_ + 1] <= '9') return err("leading zero");
        while (i_ < n_ && p_[i_] >= '0' && p_[i_] <= '9') {
            const uint64_t d = (uint64_t)(p_[i_++] - '0');
            if (v->u > (UINT64_MAX - d) / 10) v->fits = false;
            else v->u = v->u * 10 + d;
        }
        if (i_ < n_ && p_[i_] == '.') {
            v->integral = false;
            ++i_;
            if (i_ >= n_ || p_[i_] < '0' || p_[i_] > '9') return err("bad fraction");
            while (i_ < n_ && p_[i_] >= '0' && p_[i_] <= '9') ++i_;
        }
        if (i_ < n_ && (p_[i_] == 'e' || p_[i_] == 'E')) {
            v->integral = false;
            ++i_;
            if (i_ < n_ && (p_[i_] == '+' || p_[i_] == '-')) ++i_;
            if (i_ >= n_ || p_[i_] < '0' || p_[i_] > '9') return err("bad exponent");
            while (i_ < n_ && p_[i_] >= '0' && p_[i_] <= '9') ++i_;
        }
        return true;
    }
    bool value(Value* v, int depth) {
        if (depth > 32) return err("nesting too deep");
        if (i_ >= n_) return err("unexpected end");
        const char c = p_[i_];
        if (c == '{') {
            v->kind = Value::Object;
            ++i_;
            skip_ws();
            if (i_ < n_ && p_[i_] == '}') {
                ++i_;
                return true;
            }
            while (true) {
                skip_ws();
                std::pair<std::string, Value> f;
                if (!string(&f.first)) return false;
                skip_ws();
                if (i_ >= n_ || p_[i_] != ':') return err("expected ':'");
                ++i_;
                skip_ws();
                if (!value(&f.second, depth + 1)) return false;
                v->fields.push_back(std::move(f));
                skip_ws();
                if (i_ < n_ && p_[i_] == ',') {
                    ++i_;
                    continue;
                }
                if (i_ < n_ && p_[i_] == '}') {
                    ++i_;
                    return true;
                }
                return err("expected ',' or '}'");
            }
        }
        if (c == '[') {
            v->kind = Value::Array;
            ++i_;
            skip_ws();
            if (i_ < n_ && p_[i_] == ']') {
                ++i_;
                return true;
            }
            while (true) {
                skip_ws();
                Value item;
                if (!value(&item, depth + 1)) return false;
                v->items.push_back(std::move(item));
                skip_ws();
                if (i_ < n_ && p_[i_] == ',') {
                    ++i_;
                    continue;
                }
                if (i_ < n_ && p_[i_] == ']') {
                    ++i_;
                    return true;
                }
                return err("expected ',' or ']'");
            }
        }
        if (c == '"') {
            v->kind = Value::String;
            return string(&v->s);
        }
        if (c == 't') {
            v->kind = Value::Bool;
            v->b = true;
            return lit("true");
        }
        if (c == 'f') {
            v->kind = Value::Bool;
            return lit("false");
        }
        if (c == 'n') return lit("null");
        return number(v);
    }
};

}  // namespace json
}  // namespace sllm
