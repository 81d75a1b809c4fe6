// Operation parser g of App. A ("Operation Parser and Demand Prior"): the
// query text alone decides one operation category, whose demand prior (Table
// A) sets the reserve width of the allocation policy.  Procedure as the
// appendix orders it: lowercase, drop generic conversation wrappers, split
// into words, then the cue families binary decision, numerical reasoning,
// lexical readout, entity grounding in that order, the first match winning,
// general understanding otherwise.  The appendix describes the cue families
// without listing them; the phrase lists here are this library's reading.
// Host code only; no allocation beyond the query's own word list.

#include <cctype>
#include <cstring>
#include <string>
#include <vector>

#include "davet.h"

namespace davet {
int set_error(int status, const std::string& msg);
}

namespace {

// category indices of davet_demand_prior (Table A order)
enum { kCatLexical = 0, kCatNumerical = 1, kCatEntity = 2, kCatBinary = 3,
       kCatGeneral = 4 };

const char* const kWrappers[] = {
    "answer the question using a single word or phrase",
    "answer with a single word or phrase",
    "please answer the following question",
    "based on the image", "according to the image", "in the image",
    "in this image", "<image>", "question:", "answer:", "please", "briefly",
};

// yes/no interrogatives open with an auxiliary or a modal
const char* const kBinaryFirst[] = {
    "is", "are", "was", "were", "am", "do", "does", "did", "can", "could",
    "will", "would", "shall", "should", "may", "might", "must", "has", "have",
    "had", "isn't", "aren't", "wasn't", "weren't", "doesn't", "don't",
    "didn't", "can't", "won't",
};

const char* const kNumerical[] = {
    "how many", "how much", "how old", "how long", "how far", "how tall",
    "number of", "percentage", "percent", "%", "count", "total", "sum of",
    "difference", "average", "median", "ratio", "rate", "highest", "lowest",
    "maximum", "minimum", "largest", "smallest", "more than", "less than",
    "greater than", "fewer", "value of", "what value", "amount", "price",
    "cost",
};

const char* const kLexical[] = {
    "written", "write", "read", "text", "say", "says", "word", "words",
    "letter", "letters", "title", "label", "labeled", "name", "named",
    "called", "date", "when", "year", "month", "day", "time", "id",
    "identifier", "code", "number on", "address", "email", "phone", "url",
    "website", "heading", "caption", "logo", "brand", "signature", "field",
    "form",
};

const char* const kEntityFirst[] = {"who", "whom", "whose", "where"};
const char* const kEntity[] = {
    "which person", "which country", "which city", "which company",
    "which organization", "which team", "which place", "what country",
    "what city", "what company", "what organization", "what place",
    "what team",
};

// lowercase, blank out every wrapper occurrence, split into words made of
// [a-z0-9'] with '%' a word of its own
std::vector<std::string> words_of(const char* query) {
  std::string q(query);
  for (char& ch : q) ch = (char)std::tolower((unsigned char)ch);
  for (const char* w : kWrappers) {
    const size_t n = std::strlen(w);
    for (size_t at = q.find(w); at != std::string::npos; at = q.find(w, at))
      q.replace(at, n, std::string(n, ' '));
  }
  std::vector<std::string> out;
  std::string cur;
  auto flush = [&]() {
    if (!cur.empty()) out.push_back(cur);
    cur.clear();
  };
  for (char ch : q) {
    if ((ch >= 'a' && ch <= 'z') || (ch >= '0' && ch <= '9') || ch == '\'') {
      cur.push_back(ch);
    } else {
      flush();
      if (ch == '%') out.push_back("%");
    }
  }
  flush();
  return out;
}

// does the word sequence contain the phrase's words consecutively?
bool contains(const std::vector<std::string>& w, const char* phrase) {
  std::vector<std::string> p;
  std::string cur;
  for (const char* c = phrase;; ++c) {
    if (*c == ' ' || *c == '\0') {
      if (!cur.empty()) p.push_back(cur);
      cur.clear();
      if (*c == '\0') break;
    } else {
      cur.push_back(*c);
    }
  }
  if (p.empty() || p.size() > w.size()) return false;
  for (size_t i = 0; i + p.size() <= w.size(); ++i) {
    size_t k = 0;
    while (k < p.size() && w[i + k] == p[k]) ++k;
    if (k == p.size()) return true;
  }
  return false;
}

template <size_t N>
bool any_of(const std::vector<std::string>& w, const char* const (&cues)[N]) {
  for (const char* c : cues)
    if (contains(w, c)) return true;
  return false;
}

template <size_t N>
bool first_in(const std::vector<std::string>& w, const char* const (&set)[N]) {
  if (w.empty()) return false;
  for (const char* c : set)
    if (w[0] == c) return true;
  return false;
}

}  // namespace

extern "C" int davet_parse_operation(const char* query, int32_t* category) {
  if (!query || !category)
    return davet::set_error(DAVET_EINVAL, "davet_parse_operation: null argument");
  const std::vector<std::string> w = words_of(query);
  if (first_in(w, kBinaryFirst)) *category = kCatBinary;
  else if (any_of(w, kNumerical)) *category = kCatNumerical;
  else if (any_of(w, kLexical)) *category = kCatLexical;
  else if (first_in(w, kEntityFirst) || any_of(w, kEntity)) *category = kCatEntity;
  else *category = kCatGeneral;
  return DAVET_OK;
}
