"""Loader for the fixtures under tests/golden/ (hand-worked values and
tables the paper prints, each with its citation)."""

import json
import os

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def load(name: str) -> dict:
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def planner_cases():
    return load("planner_hand_examples.json")["cases"]
