"""CPU oracle of the HyperQuant codec: test infrastructure only (see oracle.py)."""
