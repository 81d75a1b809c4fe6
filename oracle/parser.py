"""Operation parser g (App. A, "Operation Parser and Demand Prior").

TEST INFRASTRUCTURE ONLY (part of the oracle): the library's own parser is
checked against this one.

g maps the query text alone to one operation category o, whose demand prior
d(o) (App. A, Table A) sets the reserve width.  The appendix fixes the
procedure -- lowercase and normalise the query, drop generic conversation
wrappers, then try the cue families in the order binary decision, numerical
reasoning, lexical readout, entity grounding and return the first match,
falling back to general understanding -- and the five representative
mappings of its example table, but not the cue lists.  The lists below are
this implementation's reading of the cue families the appendix describes.

Categories use the indices of the demand prior: 0 lexical readout,
1 numerical reasoning, 2 entity grounding, 3 binary decision, 4 general.
"""

import re

LEXICAL, NUMERICAL, ENTITY, BINARY, GENERAL = range(5)

# generic conversation wrappers removed before matching (reading)
WRAPPERS = (
    "answer the question using a single word or phrase",
    "answer with a single word or phrase",
    "please answer the following question",
    "based on the image",
    "according to the image",
    "in the image",
    "in this image",
    "<image>",
    "question:",
    "answer:",
    "please",
    "briefly",
)

# yes/no interrogatives: auxiliary- or modal-initial queries
BINARY_FIRST = {
    "is", "are", "was", "were", "am", "do", "does", "did", "can", "could",
    "will", "would", "shall", "should", "may", "might", "must", "has", "have",
    "had", "isn't", "aren't", "wasn't", "weren't", "doesn't", "don't",
    "didn't", "can't", "won't",
}

# counting, percentage, arithmetic, comparison and numerical-value requests
NUMERICAL_CUES = (
    "how many", "how much", "how old", "how long", "how far", "how tall",
    "number of", "percentage", "percent", "%", "count", "total", "sum of",
    "difference", "average", "median", "ratio", "rate", "highest", "lowest",
    "maximum", "minimum", "largest", "smallest", "more than", "less than",
    "greater than", "fewer", "value of", "what value", "amount", "price",
    "cost",
)

# text reading, dates, labels, names, titles, identifiers, document fields
LEXICAL_CUES = (
    "written", "write", "read", "text", "say", "says", "word", "words",
    "letter", "letters", "title", "label", "labeled", "name", "named",
    "called", "date", "when", "year", "month", "day", "time", "id",
    "identifier", "code", "number on", "address", "email", "phone", "url",
    "website", "heading", "caption", "logo", "brand", "signature", "field",
    "form",
)

# person, place, organisation and other entity-seeking interrogatives
ENTITY_FIRST = {"who", "whom", "whose", "where"}
ENTITY_CUES = (
    "which person", "which country", "which city", "which company",
    "which organization", "which team", "which place", "what country",
    "what city", "what company", "what organization", "what place",
    "what team",
)


def normalize(query: str) -> list:
    """Lowercase, drop the wrappers, split into words (letters, digits,
    apostrophes and '%' kept as separate tokens)."""
    q = query.lower()
    for w in WRAPPERS:
        q = q.replace(w, " ")
    return re.findall(r"[a-z0-9']+|%", q)


def _has(words: list, phrase: str) -> bool:
    p = phrase.split()
    n = len(p)
    return any(words[i:i + n] == p for i in range(len(words) - n + 1))


def parse(query: str) -> int:
    """Category of the first matching cue family in the appendix's order."""
    words = normalize(query)
    if words and words[0] in BINARY_FIRST:
        return BINARY
    if any(_has(words, c) for c in NUMERICAL_CUES):
        return NUMERICAL
    if any(_has(words, c) for c in LEXICAL_CUES):
        return LEXICAL
    if (words and words[0] in ENTITY_FIRST) or \
            any(_has(words, c) for c in ENTITY_CUES):
        return ENTITY
    return GENERAL
