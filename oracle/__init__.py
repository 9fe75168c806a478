"""CPU oracle of the cache-hit path: test infrastructure, never part of the product path."""
