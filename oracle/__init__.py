"""CPU oracle of the LCE objective -- test infrastructure, never part of the product path."""
