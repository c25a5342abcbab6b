"""Hand-worked fixtures. Each case names the passage whose rule it applies."""
import json
import os

_HERE = os.path.dirname(os.path.abspath(__file__))


def load_golden(name):
    with open(os.path.join(_HERE, name)) as f:
        data = json.load(f)
    return data["cases"]
