"""Pins of the oracle's operation parser (App. A): the appendix's example
table and its precedence rules."""

import json

import pytest

from oracle import parser


def test_paper_examples(golden_dir):
    import os
    g = json.load(open(os.path.join(golden_dir, "table_operation_examples.json")))
    for q, cat in g["examples"]:
        assert parser.parse(q) == g["categories"][cat], q


@pytest.mark.parametrize("q,cat", [
    # binary forms win over every later cue (precedence)
    ("Are there more than 5 people?", parser.BINARY),
    ("Does the title mention a date?", parser.BINARY),
    ("Can you read the label?", parser.BINARY),
    # numerical before lexical and entity
    ("What percentage of the votes did the winner get?", parser.NUMERICAL),
    ("Which year has the highest revenue?", parser.NUMERICAL),
    ("Who has the largest share?", parser.NUMERICAL),
    # lexical before entity
    ("Who wrote the text on the label?", parser.LEXICAL),
    ("When was the document signed?", parser.LEXICAL),
    ("What is the name of the street?", parser.LEXICAL),
    # entity
    ("Where was this photo taken?", parser.ENTITY),
    ("Which country is shown?", parser.ENTITY),
    # general fallback, wrappers removed before matching
    ("<image>\nDescribe the scene. Answer the question using a single word "
     "or phrase.", parser.GENERAL),
    ("", parser.GENERAL),
])
def test_precedence_and_cues(q, cat):
    assert parser.parse(q) == cat


def test_normalisation():
    assert parser.normalize("  Is THE Value   increasing?? ") == \
        ["is", "the", "value", "increasing"]
    assert parser.normalize("<image> Question: how many %?") == \
        ["how", "many", "%"]
    # cue matching is on whole words: 'account' is not 'count'
    assert parser.parse("What is the account holder doing?") == \
        parser.GENERAL
