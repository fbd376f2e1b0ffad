"""The draft-tree, tree-metadata and commit parts of the CPU oracle against what the paper and
mathematics fix (runs without a GPU)."""

import pytest

import oracle.tree_oracle as tor
from tree_pins import ALL_TREE_CHECKS


@pytest.mark.parametrize("check", ALL_TREE_CHECKS, ids=lambda f: f.__name__)
def test_tree_oracle_pin(check):
    check(tor)
